"""CPU oracle of the speculative-decoding verify step (test infrastructure).

A plain, slow, obviously-correct NumPy definition of what the GPU path computes:
the target model's forward pass over the 1+k positions of every sequence (paged-KV
attention, top-k routed mixture-of-experts, LM head) followed by the speculative
accept/resample rule. Written from the method's statement (Sec. 4.1: the serving
engine verifies k speculative tokens, zero disables; Sec. 4.1: rollout routing
replay records expert choices; Sec. 4.2: token IDs and behavior log-probabilities
are recorded at generation time; Sec. 5.3/5.4: temperature 1, no top-p/top-k) and
from the published speculative-sampling method (Leviathan, Kalman & Matias 2023;
Chen et al. 2023), in float64 unless a rounding point is part of the definition.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline``
leg may import this package. The GPU library never calls it and shares no code
with it: the only common module is ``workloads`` (seeded random inputs).
"""
from . import codecs, sampler, routing, moe, attention, model, mtp, replay, prefix  # noqa: F401
