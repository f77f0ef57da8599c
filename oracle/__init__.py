"""CPU oracle of the OPTIMA hot path (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package. The product library never does.
"""
from .optima_oracle import (hessian, damp, jacobi_scale, power_iteration, subspace_iteration, lanczos,
                            wanda_mask,
                            objective,
                            closed_form, kkt_solve, cg, rapdhg, check_decision,
                            anchor_terms, termination,
                            SolverOptions, SolveResult)

__all__ = ["hessian", "damp", "jacobi_scale", "power_iteration", "subspace_iteration", "lanczos", "wanda_mask", "objective",
           "closed_form",
           "kkt_solve", "cg", "rapdhg", "check_decision", "anchor_terms", "termination", "SolverOptions", "SolveResult"]
