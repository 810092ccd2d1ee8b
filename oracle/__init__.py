"""CPU oracle of the fingerprint forward pass -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import anything from here.  The product path (the HIP library
and its Python binding) never does, and shares no code with this package: the
one module both sides use is ``fpgen``, which only draws the seeded synthetic
inputs.

What is computed (iServe, arXiv 2501.13111): a fingerprint is the LLM cut down
to one or two hidden layers that keep the architecture's components (Sec. 1,
Sec. 5.1); the Profiler sends it dummy requests, i.e. runs prefill for the
first token and then KV-cached autoregressive decode (Sec. 5.3, Eq. 1).  The
paper never writes the layer's math; the Llama-2 style pre-norm decoder layer
(RMSNorm, rotary embedding, multi-head / grouped-query attention, SwiGLU) and
the compression menu of Sec. 3.2 (INT8 / INT4 weight-only, INT8 KV cache) are
the readings written out in ``numerics``, ``quant`` and ``layer``.

Arithmetic is float64 by default (``acc=np.float32`` is available for speed);
values are rounded to bf16 exactly at the points listed in ``layer``.

Parity status per function is stated in each module's header.  The layer as a
whole is "parity unpinned" against the model the paper profiled (the paper
gives no math and no checkpoint is available); each component is pinned by
the tests in ``tests/test_oracle_*.py``.
"""
from .numerics import bf16_round, fp16_round, rint_even  # noqa: F401
from .quant import (quant_int8_channel, dequant_int8_channel, quant_int4_g128,  # noqa: F401
                    dequant_int4_g128, pack_int4, unpack_int4, quant_kv_int8)
from .layer import (Shape, Fingerprint, rope_tables, apply_rope, rmsnorm, silu,  # noqa: F401
                    attention, argmax_first, CONFIGS)
