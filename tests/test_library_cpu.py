"""CPU: the C-ABI library loads, exports every symbol of include/*.h, and its host-side logic
(validation, conversations, occupancy, error codes) behaves as documented. No kernel runs here."""
import ctypes
import glob
import os
import re

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        src = open(h).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        names |= set(re.findall(r"\b(cs_[a-z0-9_]+)\s*\(", src))
    return names


def test_library_exports_every_declared_symbol():
    from paper_2606_01839_amd import load_library, EXPORTS
    lib = load_library()
    declared = _declared_functions()
    assert declared, "no declarations found"
    assert declared == set(EXPORTS)
    for n in declared:
        assert hasattr(lib, n), n


def test_wire_format_version_matches_the_header():
    """The binding's wire-format version is the header's (the layout the golden fixtures pin)."""
    from paper_2606_01839_amd import conserve
    src = open(os.path.join(ROOT, "include", "conserve_attn.h")).read()
    m = re.search(r"#define\s+CS_WIRE_FORMAT_VERSION\s+(\d+)", src)
    assert m and int(m.group(1)) == conserve.WIRE_FORMAT_VERSION == 1


def _pool(**kw):
    from paper_2606_01839_amd import KVPool
    args = dict(n_layers=1, n_q_heads=4, n_kv_heads=2, head_dim=64, n_pages=32, max_convs=3,
                max_pages_per_conv=8, placement_seed=1, device="cpu")
    args.update(kw)
    return KVPool(**args)


def test_descriptor_validation():
    from paper_2606_01839_amd import ConserveError, CS_EINVAL
    for bad in [dict(head_dim=96), dict(n_q_heads=6, n_kv_heads=4), dict(n_layers=0),
                dict(n_pages=0), dict(max_convs=0), dict(n_q_heads=16, n_kv_heads=1)]:
        with pytest.raises(ConserveError) as e:
            _pool(**bad)
        assert e.value.code == CS_EINVAL


def test_sizes():
    from paper_2606_01839_amd.conserve import PoolDesc, load_library
    lib = load_library()
    d = PoolDesc(32, 32, 8, 128, 256, 8192, 1000)
    assert lib.cs_pool_kv_bytes(ctypes.byref(d)) == 32 * 1000 * 8 * 2 * 16 * 128 * 2
    assert lib.cs_pool_workspace_bytes(ctypes.byref(d)) > 256 * 8192 * 4


def test_conversation_lifecycle_and_errors():
    from paper_2606_01839_amd import ConserveError, CS_ENOENT, CS_ENOMEM, CS_ESTATE, CS_EINVAL, CS_ERANGE
    p = _pool()
    a, b, c = p.conv_create(), p.conv_create(), p.conv_create()
    assert len({a, b, c}) == 3
    with pytest.raises(ConserveError) as e:
        p.conv_create()
    assert e.value.code == CS_ENOMEM
    assert p.occupancy() == (0, 32)
    assert p.conv_len(a) == 0 and len(p.conv_pages(a)) == 0
    p.conv_destroy(b)
    for fn in (lambda: p.conv_len(b), lambda: p.conv_destroy(b), lambda: p.kv_pack_size(b)):
        with pytest.raises(ConserveError) as e:
            fn()
        assert e.value.code == CS_ENOENT
    d = p.conv_create()                      # a slot is reused; the stale handle stays invalid
    assert d != b
    with pytest.raises(ConserveError) as e:
        p.conv_len(b)
    assert e.value.code == CS_ENOENT
    q1 = torch.zeros(1, 4, 64, dtype=torch.bfloat16)
    # state / argument errors are raised before anything touches a device
    with pytest.raises(ConserveError) as e:
        p.attn_extend([a], [1], 0, q1)
    assert e.value.code == CS_ESTATE
    with pytest.raises(ConserveError) as e:
        p.attn_decode_batch([a], 0, q1)
    assert e.value.code == CS_ESTATE
    q2 = torch.zeros(2, 4, 64, dtype=torch.bfloat16)
    with pytest.raises(ConserveError) as e:
        p.attn_decode_batch([a, a], 0, q2)
    assert e.value.code == CS_EINVAL
    with pytest.raises(ConserveError) as e:
        p.attn_decode_batch([a], 3, q1)
    assert e.value.code in (CS_ERANGE, CS_ESTATE)
    k = torch.zeros(1, 200, 2, 64, dtype=torch.bfloat16)
    with pytest.raises(ConserveError) as e:          # 200 tokens > 8 pages per conversation
        p.kv_append(a, k, k)
    assert e.value.code == CS_ERANGE
    assert p.conv_len(a) == 0 and p.occupancy() == (0, 32)
    with pytest.raises(ConserveError) as e:
        p.kv_unpack(torch.zeros(100, dtype=torch.uint8), 3)
    assert e.value.code in (CS_EINVAL, CS_ENOMEM)
    assert p.kv_pack_size(a) == 0
    # unknown mixed-step flags are rejected before anything is appended
    from paper_2606_01839_amd.conserve import _i32_array
    ca, cp = _i32_array([a])
    na, npp = _i32_array([1])
    kk = torch.zeros(1, 1, 2, 64, dtype=torch.bfloat16)
    qq = torch.zeros(1, 1, 4, 64, dtype=torch.bfloat16)
    rc = p.lib.cs_mixed_step(p._handle, 1, cp, npp, 0, None, kk.data_ptr(), kk.data_ptr(),
                             qq.data_ptr(), qq.data_ptr(), None, None, 2, None)
    assert rc == CS_EINVAL and p.conv_len(a) == 0
    p.close()


def test_device_calls_fail_cleanly_without_gpu():
    if torch.cuda.is_available():
        pytest.skip("has a GPU")
    from paper_2606_01839_amd import ConserveError, CS_EHIP
    p = _pool()
    a = p.conv_create()
    k = torch.zeros(1, 5, 2, 64, dtype=torch.bfloat16)
    with pytest.raises(ConserveError) as e:
        p.kv_append(a, k, k)
    assert e.value.code == CS_EHIP
    assert p.conv_len(a) == 0 and p.occupancy() == (0, 32)   # nothing committed
    p.close()
