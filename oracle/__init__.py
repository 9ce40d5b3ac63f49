"""fp64 CPU oracle of the OUTLETS hot path.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``.  The HIP library and its Python
binding never import, call or link anything here, and nothing here imports
them.  The oracle shares no code with the GPU path; the seeded input
generator (``synth``) is the only module both use, and it holds no method
arithmetic.
"""
from .formats import decode_bf16, decode_e4m3, decode_weight, decode_states  # noqa: F401
from .model import (OracleShape, OracleModel, RequestState, oracle_from_workload,  # noqa: F401
                    decode_weights, fuse, rms_norm, rope, causal_gqa_attention, silu,
                    swiglu_mlp, length_head, states_to_f64,
                    sigmoid, attention_output_gate, OracleProbe, ProbeState, probe_from_stored,
                    draft_distribution, embedded_attention_input)
from . import meta  # noqa: F401
