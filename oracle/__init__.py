"""CPU oracle for the paged-KV attention hot path -- TEST INFRASTRUCTURE ONLY.

Plain, slow, obviously-correct float64 implementations of what the GPU path computes, written from
the paper's description of serving a multi-turn conversation (prefill writes the KV cache of every
prompt token; each decode step reads the whole cache and appends one entry; later turns append new
tokens and reuse the cached prefix; the turn-1 cache is moved once to the decoder):

* ``oracle.attention`` -- causal scaled-dot-product attention over a conversation's contiguous K/V
  (no pages), for turn-1 prefill, extend and decode queries.
* ``oracle.kvwire`` -- the conversation KV store as plain concatenation, and the wire format of the
  one-time KV transfer (serialize / deserialize).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import this
package. It shares no code with the HIP library (``paper_2606_01839_amd``) and imports nothing from
it; the product path never calls it.
"""
