"""FP64 CPU oracle for the decoder-layer training hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and
its Python binding) may import, call or link anything in this package.  Only
the test-suite, the smoke check and the CPU-baseline leg of the benchmark use
it.

What it computes is the plain mathematical definition of each step, in
float64, from the float16 input values (the paper states that its backend
preserves the model computation exactly; Sec. 4.1 and Sec. 5.3):

* ``gemm``       -- C = alpha * op(A) @ op(B) + beta * C           (Sec. 4.1, FP16 GEMM backend)
                    and the column sum that is a bias gradient
* ``attention``  -- causal / GQA softmax attention forward and its
                    gradient (Sec. 4.1, Algorithm 1, Memory-resident
                    Attention Backward)
* ``swiglu``     -- SwiGLU gate of the FFN projection and its gradient
* ``norm_rope``  -- RMSNorm and rotary position embedding of the evaluated
                    models (Sec. 6.1) and their gradients
* ``layer``      -- one decoder layer forward + backward composed of the above
                    (optionally with the models' RMSNorm and rotary embedding)
* ``pipeline``   -- the non-interleaved 1F1B schedule as a discrete-event
                    simulation (makespan, resident micro-batches per stage;
                    Sec. 4.3-4.4), the reference for the planner

No blocking, fusion, online softmax or reordering: a reader can check each
function against the definitions by eye.  Library primitives used as single
steps: numpy's float64 matmul, exp, log and reductions.

Every function here is pinned by the CPU tests in ``tests/test_oracle_*.py``
(brute force, closed forms, finite differences, invariants, hand-derived
worked examples under ``tests/golden/``).
"""

from .gemm import gemm, gemm_entries, column_sum
from .attention import attn_fwd, attn_bwd, attn_head_fwd, attn_head_bwd
from .swiglu import silu, swiglu_fwd, swiglu_bwd
from .norm_rope import rmsnorm_fwd, rmsnorm_bwd, rope_angles, rope_fwd, rope_bwd
from .layer import LayerShape, LayerNorms, layer_fwd, layer_bwd, layer_flops
from .pipeline import stage_order, simulate_1f1b

__all__ = [
    "gemm", "gemm_entries", "column_sum",
    "attn_fwd", "attn_bwd", "attn_head_fwd", "attn_head_bwd",
    "silu", "swiglu_fwd", "swiglu_bwd",
    "rmsnorm_fwd", "rmsnorm_bwd", "rope_angles", "rope_fwd", "rope_bwd",
    "LayerShape", "LayerNorms", "layer_fwd", "layer_bwd", "layer_flops",
    "stage_order", "simulate_1f1b",
]
