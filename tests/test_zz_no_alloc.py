"""GPU: the allocation-free decode entry point (cs_attn_decode_batch_noalloc) against
cs_attn_decode_batch, through the C ABI.

Two calls in a row on one pool, the second with a smaller batch, each bitwise equal to the
existing entry point's output (same kernels; only the partial records' buffer differs) and within
the attention tolerance of the fp64 oracle; a direct-path batch (every conversation one work item,
no partial records); and a batch whose partial records exceed the static scratch, which is refused
with CS_ENOMEM before anything is launched.
"""
import numpy as np
import pytest
import torch

from oracle.attention import attend_last
from tests.helpers import assert_close, f64, kv_tokens, q_tokens

pytestmark = pytest.mark.gpu

SEED = 4242
HQ, HKV, D = 32, 8, 128


def _pool(lens, max_convs=16):
    from paper_2606_01839_amd import KVPool
    pool = KVPool(1, HQ, HKV, D, n_pages=sum((L + 15) // 16 for L in lens) + 8, max_convs=max_convs,
                  max_pages_per_conv=4096, placement_seed=9, device="cuda")
    convs, kvs = [], []
    for i, L in enumerate(lens):
        c = pool.conv_create()
        k, v = kv_tokens(SEED, i, 1, 0, L, HKV, D)
        pool.kv_append(c, k.cuda(), v.cuda())
        convs.append(c)
        kvs.append((k, v))
    return pool, convs, kvs


def _queries(idx, lens):
    return torch.cat([q_tokens(SEED, i, 0, lens[i] - 1, 1, HQ, D) for i in idx]).cuda()


def test_noalloc_decode_matches_decode_batch_twice():
    lens = [9000, 20000, 3000, 700, 1, 1100]
    print("no-alloc decode: lens", lens, flush=True)
    pool, convs, kvs = _pool(lens)
    for idx in ([0, 1, 2, 3, 4, 5], [3, 4, 2]):          # second call: a smaller batch
        sel = [convs[i] for i in idx]
        q = _queries(idx, lens)
        out = torch.full((len(idx), HQ, D), float("nan"), dtype=torch.bfloat16, device="cuda")
        pool.attn_decode_batch_noalloc(sel, 0, q, out)
        want = pool.attn_decode_batch(sel, 0, q)
        torch.cuda.synchronize()
        assert torch.equal(out, want), f"batch {idx}: no-alloc output differs from cs_attn_decode_batch"
        for r, i in enumerate(idx):
            k, v = kvs[i]
            ref = attend_last(f64(q[r:r + 1].cpu()), f64(k[0]), f64(v[0]))
            assert_close(out[r:r + 1], ref, f"no-alloc decode conv {i} (L {lens[i]})")
    pool.close()


def test_noalloc_decode_direct_path():
    lens = [1, 17, 500, 1024]                             # every conversation one work item
    print("no-alloc decode direct: lens", lens, flush=True)
    pool, convs, kvs = _pool(lens)
    q = _queries(range(len(lens)), lens)
    out = torch.empty((len(lens), HQ, D), dtype=torch.bfloat16, device="cuda")
    pool.attn_decode_batch_noalloc(convs, 0, q, out)
    want = pool.attn_decode_batch(convs, 0, q)
    torch.cuda.synchronize()
    assert torch.equal(out, want)
    pool.close()


def test_noalloc_decode_refuses_partials_beyond_the_scratch():
    """997 work items x 32 query heads x 132 floats > 4,194,304 floats: CS_ENOMEM, nothing written."""
    from paper_2606_01839_amd import ConserveError, CS_ENOMEM
    lens = [1] * 995 + [9000]
    print("no-alloc decode: oversized batch", flush=True)
    from paper_2606_01839_amd import KVPool
    pool = KVPool(1, HQ, HKV, D, n_pages=995 + 563 + 8, max_convs=996, max_pages_per_conv=1024,
                  placement_seed=3, device="cuda")
    convs = [pool.conv_create() for _ in lens]
    k = torch.zeros((1, sum(lens), HKV, D), dtype=torch.bfloat16, device="cuda")
    pool.kv_append_batch(convs, lens, k, k)
    q = torch.zeros((len(lens), HQ, D), dtype=torch.bfloat16, device="cuda")
    out = torch.full((len(lens), HQ, D), 7.0, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ConserveError) as e:
        pool.attn_decode_batch_noalloc(convs, 0, q, out)
    assert e.value.code == CS_ENOMEM and "static scratch" in str(e.value)
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
    # the same batch through the pool's workspace works
    pool.attn_decode_batch(convs, 0, q, out)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(out.float()).all())
    pool.close()
