"""The oracle: a plain, slow float64 CPU reference of the hot path.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package. The product
library (``paper_1711_03016_amd``) never imports, links or runs it, and the two
share no code: the oracle interprets an SSA tensor IR with NumPy in float64 and
differentiates it by adjoint code generation (DLVM §3.1.3); the product runs
hand-written HIP kernels.

Parity status: every function here is pinned by CPU tests against values that
do not come from the oracle itself (finite differences, closed forms,
invariants, special cases, an independent library autograd).
"""
from .ad import adce, count_ops, differentiate, simplify_algebra  # noqa: F401
from .bf16 import bf16_bits, round_to_bf16  # noqa: F401
from .ir import Function, evaluate  # noqa: F401
from .mlp import (MlpSpec, apply_act, chain8, dense_forward, dense_vjp_input,  # noqa: F401
                  dense_vjp_params, gemm, mlp_forward, mlp_gradient, mlp_vjp, sgd_bf16,
                  sgd_f32, softmax_xent)
from .rnn import RnnSpec, rnn_forward, rnn_vjp  # noqa: F401
from .chain import chain_order, chain_product, chain_product_in_order, parenthesisation  # noqa: F401
