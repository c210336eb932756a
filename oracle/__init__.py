"""CPU oracle for FastVLM's greedy self-speculative decoding (arXiv 2510.22641).

TEST INFRASTRUCTURE ONLY.  This package is the slow, plain float64 reference that the
device path is checked against.  Only the tests, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it; the product path never does, and it
shares no code with the HIP library (the seeded input generators in ``synth`` serve both).

Contents
  ops.py     norms, activations, relative-position buckets, rotary embedding, softmax attention
  model.py   the decoder (T5-v1.1-style with cross-attention, or LLaMA-2-style), the imitation
             network and the shared LM head g, evaluated position by position
  decode.py  prefill, full-model greedy decoding, Algorithm 1 (self-speculative imitation
             decoding, greedy) and a replay mode that follows a device run's token stream
  sampling.py  the sampling variant of the loop (speculative sampling, uniforms as inputs),
             plain sampling from the full model, and its replay mode

Precision: float64 throughout, on the float32 (bf16-representable, in bf16 workloads) values
produced by ``synth``.

Pinning: every function is checked in tests/test_oracle_*.py against closed forms,
invariants, brute force on tiny inputs or library routines; see each module's header.
Parity unpinned: the imitation network's exact form (the paper names two fully connected
layers and one layer norm but prints no numbers) and the synthetic initialisation choices;
their arithmetic is pinned by closed-form special cases, the reading itself is not.
"""
