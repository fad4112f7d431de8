"""Float64 CPU oracle for sink-anchored windowed-KV frame attention.

TEST INFRASTRUCTURE ONLY. Nothing in the product path (the HIP library and its
Python binding) imports, links or runs anything here; only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may.
The oracle shares no code with the GPU path: no kernels, headers, tables or
pre/post-processing.  The only thing both sides consume is the seeded input
generator in ``workload/``, which holds none of the method's arithmetic.

Modules
-------
``windowed_attention``
    The attention state machine of Metronome (arXiv 2607.02640) §4.1 and
    App. A: each session retains its first S tokens (the pinned sinks) plus the
    last W tokens, and every query attends to sinks ∪ window under causality.
    Plain definition, float64, explicit retained-set dictionaries.
``index_model``
    The pool/block/ring index arithmetic (block pinning of App. A "Sink half",
    free-behind-window of App. A "Window half", the pool-fill law of §3.1 Eq. 1)
    as an independent pure-Python model, compared bit-exactly with the library.
``admission``
    The deadline-aware admission loop of §4.2 (AIMD on the per-frame latency:
    multiplicative cut near the target, additive probe with headroom, clean
    rejection beyond the cap), compared call by call with the library's
    host-only controller.
``fp8_kv``
    The OCP E4M3 codec and the per-(token, head) power-of-two scale rule of
    the FP8 KV cache (per-token KV reduction composes with the window, §4.1
    and §6), written from the format's definition; ``OracleSession`` applies
    it to every stored row when ``kv_quant="fp8_e4m3"``.

Parity status of each function is stated in its module header.
"""
