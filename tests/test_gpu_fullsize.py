"""GPU parity at the benchmark sizes, in the launch configuration bench.py times.

* decode batch (64 conversations, 8k-32k context, per-head scales): every conversation's output.
* extend (16 conversations, prefix 16k-64k, chunk ~1k): sampled query rows of every conversation --
  first and last row of each chunk, page- and tile-boundary rows, seeded random rows.
* turn-1 prefill (8 conversations, 32k-128k): sampled rows, same rule.
The oracle's inputs are the seeded generator's values; the device-generated copies used here are
checked bit for bit against host generation on sampled rows first.
"""
import numpy as np
import pytest
import torch

import bench
from oracle.attention import attend_rows
from synth import values as sv
from synth.traces import DecodeBatch, ExtendBatch, PrefillTransfer, KIND_K, KIND_V
from tests.helpers import assert_close

pytestmark = pytest.mark.gpu


def _check_rows_equal_host(dev, seed, conv, kind, H, d, positions, start=0, scale=None):
    key = sv.mix_key(seed, conv, kind, 0)
    for p in positions:
        host = sv.bf16_tensor(key, (1, H, d), head_scale=scale, start=p * H * d)
        assert torch.equal(dev[p - start].cpu(), host[0]), (conv, kind, p)


def _sample_rows(n, P, rng, extra=3):
    rows = {0, n - 1}
    for i in range(n):                      # first page and first tile boundary inside the chunk
        if (P + i) % 16 == 0:
            rows.add(i)
            break
    for i in range(n):
        if (P + i) % 64 == 63:
            rows.add(i)
            break
    rows |= set(int(x) for x in rng.integers(0, n, size=extra))
    return sorted(r for r in rows if 0 <= r < n)


def test_decode_batch_full_size():
    tr = DecodeBatch()
    sk, svs = tr.head_scales()
    pool, convs, lens, kv_dev, q = bench.make_decode_case(tr)
    out = pool.attn_decode_batch(convs, 0, q)
    torch.cuda.synchronize()
    sh = tr.shape
    rng = np.random.default_rng(0)
    for b in range(len(lens)):
        L = int(lens[b])
        pos = [0, L - 1, int(rng.integers(0, L))]
        _check_rows_equal_host(kv_dev[b][0], tr.seed, b, KIND_K, sh.n_kv_heads, sh.head_dim, pos, scale=sk)
        _check_rows_equal_host(kv_dev[b][1], tr.seed, b, KIND_V, sh.n_kv_heads, sh.head_dim, pos, scale=svs)
    got, ref = [], []
    for b in range(len(lens)):
        k = sv.bf16_to_f64(kv_dev[b][0])
        v = sv.bf16_to_f64(kv_dev[b][1])
        ref.append(attend_rows(sv.bf16_to_f64(q[b:b + 1]), [int(lens[b]) - 1], k, v))
        got.append(out[b:b + 1])
    assert_close(torch.cat(got), np.concatenate(ref), "decode batch, all 64 conversations")
    pool.close()


def test_extend_full_size_sampled_rows():
    tr = ExtendBatch()
    sh = tr.shape
    pool, convs, prefix, chunk, kcat, vcat, q = bench.make_extend_case(tr)
    pool.kv_append_batch(convs, chunk, kcat, vcat)
    out = pool.attn_extend(convs, chunk, 0, q)
    torch.cuda.synchronize()
    rng = np.random.default_rng(1)
    got, ref = [], []
    row0 = 0
    for b in range(tr.n_convs):
        P, n = int(prefix[b]), int(chunk[b])
        k, v = bench.gen_kv(tr.seed, b, 0, P + n, sh.n_kv_heads, sh.head_dim)
        _check_rows_equal_host(k, tr.seed, b, KIND_K, sh.n_kv_heads, sh.head_dim, [0, P - 1, P + n - 1])
        kf, vf = sv.bf16_to_f64(k), sv.bf16_to_f64(v)
        rows = _sample_rows(n, P, rng)
        qr = sv.bf16_to_f64(q[row0:row0 + n][rows])
        ref.append(attend_rows(qr, [P + i for i in rows], kf, vf))
        got.append(out[row0:row0 + n][rows])
        row0 += n
    assert_close(torch.cat(got), np.concatenate(ref), "extend, sampled rows of 16 conversations")
    pool.close()


def test_turn1_prefill_full_size_sampled_rows():
    tr = PrefillTransfer()
    sh = tr.shape
    pool, convs, lens, q = bench.make_prefill_case(tr)
    out = pool.attn_prefill_turn1(convs, lens, 0, q)
    torch.cuda.synchronize()
    rng = np.random.default_rng(2)
    got, ref = [], []
    row0 = 0
    for b, L in enumerate(lens):
        L = int(L)
        k, v = bench.gen_kv(tr.seed, b, 0, L, sh.n_kv_heads, sh.head_dim)
        _check_rows_equal_host(v, tr.seed, b, KIND_V, sh.n_kv_heads, sh.head_dim, [0, L // 2, L - 1])
        kf, vf = sv.bf16_to_f64(k), sv.bf16_to_f64(v)
        rows = sorted(set(_sample_rows(L, 0, rng)) | {1, 15, 16, 63, 64})
        ref.append(attend_rows(sv.bf16_to_f64(q[row0:row0 + L][rows]), rows, kf, vf))
        got.append(out[row0:row0 + L][rows])
        row0 += L
        del k, v, kf, vf
    assert_close(torch.cat(got), np.concatenate(ref), "turn-1 prefill, sampled rows of 8 conversations")
    pool.close()


def test_turn1_transfer_full_size_bit_exact():
    """The one-time transfer of the whole turn-1 batch (8 conversations, 32k-128k tokens): pack ->
    unpack into a pool with another placement -> pack again is byte-identical; the destination's
    page tables are valid; sampled wire pages equal the oracle's serialization of the generator's
    tokens (first, second, last two and seeded random pages of every conversation)."""
    from oracle import kvwire
    from paper_2606_01839_amd import KVPool
    tr = PrefillTransfer()
    sh = tr.shape
    hkv, d = sh.n_kv_heads, sh.head_dim
    pool, convs, lens, q = bench.make_prefill_case(tr)
    del q
    wires = [pool.kv_pack(c) for c in convs]
    dst = KVPool(1, sh.n_q_heads, hkv, d, n_pages=pool.desc.n_pages, max_convs=tr.n_convs,
                 max_pages_per_conv=bench.pages_for(tr.hi), placement_seed=tr.dst_seed)
    dconvs = [dst.kv_unpack(w, int(L)) for w, L in zip(wires, lens)]
    torch.cuda.synchronize()
    seen = set()
    for c, w, L in zip(dconvs, wires, lens):
        assert torch.equal(dst.kv_pack(c), w)
        pages = dst.conv_pages(c)
        assert len(pages) == bench.pages_for(int(L)) and all(0 <= p < dst.desc.n_pages for p in pages)
        assert not (seen & set(pages))
        seen |= set(pages)
    assert dst.occupancy()[0] == len(seen)
    rng = np.random.default_rng(3)
    block = hkv * 2 * 16 * d                       # uint16 elements per logical page (one layer)
    for b, (w, L) in enumerate(zip(wires, lens)):
        L = int(L)
        n_pg = bench.pages_for(L)
        wire = w.cpu().numpy().view(np.uint16)
        for p in sorted({0, 1, n_pg - 2, n_pg - 1} | set(int(x) for x in rng.integers(0, n_pg, size=5))):
            t0, t1 = 16 * p, min(L, 16 * p + 16)
            k, v = bench.gen_kv(tr.seed, b, t0, t1 - t0, hkv, d, device="cpu")
            want = kvwire.serialize(sv.bf16_bits(k)[None], sv.bf16_bits(v)[None])
            assert np.array_equal(wire[p * block:(p + 1) * block], want), (b, p)
    pool.close()
    dst.close()
