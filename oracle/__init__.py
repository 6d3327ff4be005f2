"""Plain fp64 CPU oracle of the DraftAttention2 hot path.

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import it. The GPU library never
calls into it, and it shares no code with the GPU library.

Modules follow the paper's order of operations:

* ``formats``   - E4M3 / E2M1 / INT8 casts (quantization-format appendix).
* ``partition`` - spatial regions and slot maps (fused preparation section,
                  ragged-padding equation; here fixed 8x8 tiles).
* ``draft``     - average / max pooled descriptors and the draft map
                  (descriptor equation, Definition 3.1).
* ``rank``      - integer quotas and the shared ranking (Algorithm 1).
* ``encode``    - INT8, E4M3 and NVFP4 operand encodings (format appendix,
                  NVFP4 quantization equation).
* ``attention`` - phased attention with shared online-softmax state
                  (precision-state-conversion equation, phased-execution
                  appendix), dense reference and error-bound diagnostics
                  (Lemma 3.2).
* ``pipeline``  - the four stages end to end.
"""
