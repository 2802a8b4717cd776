"""GPU: error paths after validation, forced from the host with cs_debug_fail_launches (the failing
launch reports CS_EHIP without launching anything, so no kernel ever faults).

* A failed append changes no length, page list or occupancy, also when an earlier launch of the
  same append already ran (an append of more than one upload group); appending the same tokens
  again afterwards gives the oracle's attention output.
* A failed attention call changes nothing; the next call works.
* cs_mixed_step whose attention launch fails has completed its append (documented behaviour).
"""
import numpy as np
import pytest
import torch

from oracle.attention import attend_last
from tests.helpers import assert_close, f64, kv_tokens, q_tokens

pytestmark = pytest.mark.gpu

SEED = 515


def _pool(hq, hkv, d, n_pages, max_pages=4096, n_layers=1, seed=3):
    from paper_2606_01839_amd import KVPool
    return KVPool(n_layers, hq, hkv, d, n_pages=n_pages, max_convs=8, max_pages_per_conv=max_pages,
                  placement_seed=seed, device="cuda")


def _state(pool, convs):
    return [pool.conv_len(c) for c in convs], [pool.conv_pages(c).tolist() for c in convs], pool.occupancy()


def test_failed_append_changes_nothing_then_succeeds():
    from paper_2606_01839_amd import ConserveError, CS_EHIP
    hq, hkv, d = 8, 2, 64
    print("failed append: single and batched", flush=True)
    pool = _pool(hq, hkv, d, 64)
    a, b = pool.conv_create(), pool.conv_create()
    ka, va = kv_tokens(SEED, 0, 1, 0, 60, hkv, d)
    kb, vb = kv_tokens(SEED, 1, 1, 0, 45, hkv, d)
    pool.kv_append(a, ka[:, :20].contiguous().cuda(), va[:, :20].contiguous().cuda())
    pool.kv_append(b, kb[:, :5].contiguous().cuda(), vb[:, :5].contiguous().cuda())
    before = _state(pool, [a, b])
    pool.debug_fail_launches(0)
    with pytest.raises(ConserveError) as e:
        pool.kv_append(a, ka[:, 20:].contiguous().cuda(), va[:, 20:].contiguous().cuda())
    assert e.value.code == CS_EHIP and "injected" in str(e.value)
    with pytest.raises(ConserveError):
        pool.kv_append_batch([a, b], [40, 40], torch.cat([ka[:, 20:], kb[:, 5:]], 1).contiguous().cuda(),
                             torch.cat([va[:, 20:], vb[:, 5:]], 1).contiguous().cuda())
    assert _state(pool, [a, b]) == before
    pool.debug_fail_launches(-1)
    pool.kv_append_batch([a, b], [40, 40], torch.cat([ka[:, 20:], kb[:, 5:]], 1).contiguous().cuda(),
                         torch.cat([va[:, 20:], vb[:, 5:]], 1).contiguous().cuda())
    q = torch.cat([q_tokens(SEED, 0, 0, 59, 1, hq, d), q_tokens(SEED, 1, 0, 44, 1, hq, d)]).cuda()
    out = pool.attn_decode_batch([a, b], 0, q)
    torch.cuda.synchronize()
    assert_close(out[0:1], attend_last(f64(q[0:1].cpu()), f64(ka[0]), f64(va[0])), "conv a after the retry")
    assert_close(out[1:2], attend_last(f64(q[1:2].cpu()), f64(kb[0]), f64(vb[0])), "conv b after the retry")
    pool.close()


def test_append_failing_in_its_second_launch_rolls_back():
    """65,537 page chunks need two uploads and two launches; the second fails after the first ran."""
    from paper_2606_01839_amd import ConserveError, CS_EHIP
    hq, hkv, d = 2, 1, 64
    L0, n = 8, 65536 * 16 + 1
    print("failed append in its second launch", flush=True)
    pool = _pool(hq, hkv, d, 65540, max_pages=65540)
    c = pool.conv_create()
    k, v = kv_tokens(SEED, 7, 1, 0, L0 + n, hkv, d)
    pool.kv_append(c, k[:, :L0].contiguous().cuda(), v[:, :L0].contiguous().cuda())
    before = _state(pool, [c])
    kn, vn = k[:, L0:].contiguous().cuda(), v[:, L0:].contiguous().cuda()
    pool.debug_fail_launches(1)
    with pytest.raises(ConserveError) as e:
        pool.kv_append(c, kn, vn)
    assert e.value.code == CS_EHIP
    assert _state(pool, [c]) == before
    pool.debug_fail_launches(-1)
    pool.kv_append(c, kn, vn)
    q = q_tokens(SEED, 7, 0, L0 + n - 1, 1, hq, d).cuda()
    out = pool.attn_decode_batch([c], 0, q)
    torch.cuda.synchronize()
    assert_close(out, attend_last(f64(q.cpu()), f64(k[0]), f64(v[0])), "after the retried long append")
    pool.close()


def test_failed_attention_and_mixed_step():
    from paper_2606_01839_amd import ConserveError, CS_EHIP
    hq, hkv, d = 32, 8, 128
    print("failed attention and mixed step", flush=True)
    pool = _pool(hq, hkv, d, 64)
    c = pool.conv_create()
    k, v = kv_tokens(SEED, 3, 1, 0, 301, hkv, d)
    pool.kv_append(c, k[:, :300].contiguous().cuda(), v[:, :300].contiguous().cuda())
    q = q_tokens(SEED, 3, 0, 299, 1, hq, d).cuda()
    before = _state(pool, [c])
    pool.debug_fail_launches(0)
    for call in (lambda: pool.attn_decode_batch([c], 0, q), lambda: pool.attn_extend([c], [1], 0, q)):
        with pytest.raises(ConserveError) as e:
            call()
        assert e.value.code == CS_EHIP
    assert _state(pool, [c]) == before
    # mixed step: its append launch runs, the first attention launch fails
    pool.debug_fail_launches(1)
    q2 = q_tokens(SEED, 3, 0, 300, 1, hq, d).cuda()
    with pytest.raises(ConserveError) as e:
        pool.mixed_step([], [], [c], k[:, 300:].contiguous().cuda(), v[:, 300:].contiguous().cuda(),
                        q_dec=q2[None].contiguous())
    assert e.value.code == CS_EHIP and pool.conv_len(c) == 301
    pool.debug_fail_launches(-1)
    out = pool.attn_decode_batch([c], 0, q2)
    torch.cuda.synchronize()
    assert_close(out, attend_last(f64(q2.cpu()), f64(k[0]), f64(v[0])), "decode after the failed mixed step")
    pool.close()
