"""Plain fp64 CPU oracle for incremental chunked-prefill attention over a paged KV cache.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import anything from this package.  The
GPU library under ``paper_2604_16395_amd/`` never imports it, and this package
imports nothing from the GPU library: the two share no code.

What it computes (Stream2LLM, arXiv 2604.16395):

* the prefill of a request produces one key/value pair per token and keeps them as the
  KV cache (Sec. 2.1); the cache is split into fixed blocks of k tokens whose physical
  placement is arbitrary, and attention at position t reads every block covering
  positions up to t (Sec. 2.2);
* a streamed request that already holds ``num_computed_tokens`` cached tokens resumes
  prefill from that point (Sec. 4.2), which in append mode means a new chunk of C
  tokens is added after the P cached ones (Sec. 5.1, the append/update listing).

Modules:

* :mod:`oracle.fp8_e4m3`  - OCP FP8 E4M3 (``e4m3fn``) decode table and RNE/satfinite encoder.
* :mod:`oracle.paged_kv`  - page/slot addressing, page append (scatter) and gather.
* :mod:`oracle.attention` - chunk attention by definition (per-row loops and a blocked
  two-pass form), brute-force full causal attention, and the log-sum-exp merge.

Every function works in float64 (bf16 and fp8 values convert to float64 exactly).
Parity status of each function is recorded in its docstring; all are pinned by the
``-m "not gpu"`` tests in ``tests/test_oracle_*.py``.
"""
