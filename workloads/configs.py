"""Layer configurations for the synthetic workloads.

Each configuration describes one pruned linear layer: the calibration token
matrix X (n_tok x d, streamed in sequences of `chunk` tokens, as in the
incremental Hessian of Section 3.4), the dense weight W0 (n_cols x d, one QP per
row, i.e. per output column of the paper's d_in x d_out weight, Eq. (3)), and
the mask recipe. The shapes and value distributions stand in for the paper's
128 x 2048-token C4 calibration set (Appendix D, Table 8); no C4 data is used.

This module holds no arithmetic of the method: it only names sizes and seeds.
"""
from dataclasses import dataclass, field, replace


@dataclass(frozen=True)
class LayerConfig:
    name: str
    cfg_id: int            # first word of every seed sequence of this layer
    d: int                 # d_in: QP dimension and Hessian side
    n_cols: int            # d_out: number of column QPs
    n_tok: int             # calibration tokens (sequences x sequence length)
    chunk: int             # tokens per calibration sequence
    x_dtype: str           # "f32" or "bf16": storage type of X
    w_dtype: str           # "f32" or "bf16": storage type of W0 (values only)
    w_std: float           # W0 ~ N(0, w_std^2)
    x_recipe: str          # "ar1" | "lognormal" | "student_t_outliers" | "silu_gated"
    mask_kind: str         # "unstructured" | "2:4"
    sparsity: float        # fraction pruned per column (unstructured)
    rel_damp: float = 0.01  # lambda = rel_damp * mean(diag(X^T X))
    n_outliers: int = 8
    outlier_scale: float = 50.0
    t_dof: int = 4
    tensor_offset: int = 0  # added to tensor ids (block matrices use 10*k)

    @property
    def n_chunks(self) -> int:
        return (self.n_tok + self.chunk - 1) // self.chunk

    def with_tokens(self, n_tok: int) -> "LayerConfig":
        """Same layer with fewer (or more) calibration tokens."""
        return replace(self, n_tok=n_tok)

    def with_cols(self, n_cols: int) -> "LayerConfig":
        return replace(self, n_cols=n_cols)


# Tensor ids inside a layer's seed sequence [cfg_id, tensor_id, index].
TENSOR_X = 0
TENSOR_W0 = 1
TENSOR_OUTLIERS = 2
TENSOR_SCALES = 3
TENSOR_V0 = 4          # start vector of the power iteration
TENSOR_GATE = 5        # second factor of the SiLU-gated activations

TINY = LayerConfig(
    name="tiny", cfg_id=0, d=128, n_cols=64, n_tok=512, chunk=512,
    x_dtype="f32", w_dtype="f32", w_std=0.02, x_recipe="ar1",
    mask_kind="unstructured", sparsity=0.5)

GPT2_FC = LayerConfig(
    name="gpt2_fc", cfg_id=1, d=768, n_cols=3072, n_tok=128 * 2048, chunk=2048,
    x_dtype="bf16", w_dtype="bf16", w_std=0.02, x_recipe="lognormal",
    mask_kind="unstructured", sparsity=0.5)

Q_PROJ = LayerConfig(
    name="q_proj", cfg_id=2, d=4096, n_cols=4096, n_tok=128 * 2048, chunk=2048,
    x_dtype="bf16", w_dtype="bf16", w_std=0.015, x_recipe="student_t_outliers",
    mask_kind="2:4", sparsity=0.5)

DOWN_PROJ = LayerConfig(
    name="down_proj", cfg_id=3, d=14336, n_cols=4096, n_tok=128 * 2048, chunk=2048,
    x_dtype="bf16", w_dtype="bf16", w_std=0.015, x_recipe="silu_gated",
    mask_kind="unstructured", sparsity=0.6)

CONFIGS = {c.name: c for c in (TINY, GPT2_FC, Q_PROJ, DOWN_PROJ)}

# The Llama-3-8B-shaped decoder block, streamed layer by layer: four
# calibration streams (the inputs of q/k/v, of o, of gate/up and of down; the
# first three follow the q_proj recipe, the last the down_proj recipe), 128 x
# 2048 tokens each, and seven weight matrices with 50 % unstructured masks.
# Streams draw their tokens under cfg_id 4 with tensor ids offset by 10 k;
# each matrix draws its W0 with an offset of its own (40, 50, ...).
_BLOCK_STREAM_RECIPES = (
    ("qkv_in", 4096, "student_t_outliers"),
    ("o_in", 4096, "student_t_outliers"),
    ("gate_up_in", 4096, "student_t_outliers"),
    ("down_in", 14336, "silu_gated"),
)
BLOCK_STREAMS = {
    name: LayerConfig(
        name=f"block_{name}", cfg_id=4, d=d, n_cols=0, n_tok=128 * 2048, chunk=2048,
        x_dtype="bf16", w_dtype="bf16", w_std=0.015, x_recipe=recipe,
        mask_kind="unstructured", sparsity=0.5, tensor_offset=10 * k)
    for k, (name, d, recipe) in enumerate(_BLOCK_STREAM_RECIPES)
}
# (matrix, stream, output columns)
_BLOCK_MATRICES = (("q_proj", "qkv_in", 4096), ("k_proj", "qkv_in", 1024),
                   ("v_proj", "qkv_in", 1024), ("o_proj", "o_in", 4096),
                   ("gate_proj", "gate_up_in", 14336), ("up_proj", "gate_up_in", 14336),
                   ("down_proj", "down_in", 4096))
BLOCK_LAYERS = tuple(
    (replace(BLOCK_STREAMS[stream], name=f"block_{name}", n_cols=cols,
             tensor_offset=40 + 10 * i), stream)
    for i, (name, stream, cols) in enumerate(_BLOCK_MATRICES))


@dataclass(frozen=True)
class SolverSettings:
    """Solver budgets used with the configurations (Appendix D, Table 8)."""
    paper_eps: float = 0.01        # relative and absolute tolerance
    paper_max_iters: int = 100_000
    check_every: int = 64
    tiny_fixed_iters: int = 1000

# A chain of four 4096 x 4096 linear layers with SiLU between them, for the
# layer loop of Algorithm 1 (each layer is pruned on the pruned outputs of the
# one before). Its input stream follows the q_proj recipe (128 x 2048 bf16
# tokens, seeds of its own); the weights are N(0, 0.015^2) with 50 %
# unstructured masks.
CHAIN_STREAM = LayerConfig(
    name="chain_in", cfg_id=5, d=4096, n_cols=0, n_tok=128 * 2048, chunk=2048,
    x_dtype="bf16", w_dtype="bf16", w_std=0.015, x_recipe="student_t_outliers",
    mask_kind="unstructured", sparsity=0.5)

CHAIN_LAYERS = tuple(
    replace(CHAIN_STREAM, name=f"chain_l{i}", n_cols=4096, tensor_offset=10 * (i + 1))
    for i in range(4))
