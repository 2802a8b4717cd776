"""Pins of the CPU oracle against facts fixed outside it (no GPU).

Each pin is chosen so that a plausible mistake in the oracle fails at least one test:
* brute force (independent pure-Python loops, math.fsum)   -> any arithmetic slip
* hand-worked example (tests/golden)                        -> scale, causal diagonal, order
* Q = 0 closed form (running mean of V)                     -> off-by-one in the causal mask
* L = 1 and concentration limits                            -> softmax normalisation / indexing
* GQA == MHA with repeated KV                               -> head mapping
* chunked extend == one-shot prefill, decode == last row    -> query positions of extend/decode
"""
import math
import os

import numpy as np
import pytest

from oracle.attention import attend_last, attend_rows, kv_head_of, weights
from oracle import kvwire

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def brute_attend(q, k, v):
    """Pure-Python causal attention, last n positions, written independently of the oracle."""
    n, hq, d = len(q), len(q[0]), len(q[0][0])
    L, hkv = len(k), len(k[0])
    grp = hq // hkv
    out = [[[0.0] * d for _ in range(hq)] for _ in range(n)]
    for i in range(n):
        p = L - n + i
        for h in range(hq):
            g = h // grp
            s = [math.fsum(q[i][h][e] * k[j][g][e] for e in range(d)) / math.sqrt(d)
                 for j in range(p + 1)]
            m = max(s)
            w = [math.exp(x - m) for x in s]
            z = math.fsum(w)
            for e in range(d):
                out[i][h][e] = math.fsum(w[j] * v[j][g][e] for j in range(p + 1)) / z
    return np.array(out)


def rand_case(rng, L, n, hq, hkv, d, scale=1.0):
    q = rng.standard_normal((n, hq, d)) * scale
    k = rng.standard_normal((L, hkv, d)) * scale
    v = rng.standard_normal((L, hkv, d))
    return q, k, v


@pytest.mark.parametrize("seed", range(12))
def test_oracle_matches_brute_force(seed):
    rng = np.random.default_rng(seed)
    hq, hkv = [(1, 1), (2, 1), (4, 2), (4, 1), (6, 3)][seed % 5]
    d = [4, 8, 16][seed % 3]
    L = int(rng.integers(1, 41))
    n = int(rng.integers(1, L + 1))
    q, k, v = rand_case(rng, L, n, hq, hkv, d, scale=1.5)
    got = attend_last(q, k, v)
    ref = brute_attend(q.tolist(), k.tolist(), v.tolist())
    assert got.shape == ref.shape
    err = np.abs(got - ref).max() / max(1e-300, np.abs(ref).max())
    assert err <= 1e-12, err


def _parse_golden_attention():
    rows = {"k": {}, "v": {}, "q": {}, "o": {}}
    env = {"LN2": math.log(2.0), "LN3": math.log(3.0), "LN4": math.log(4.0)}
    with open(os.path.join(GOLDEN, "attention_worked_example.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            tag, idx, *vals = line.split()
            rows[tag][int(idx)] = [float(eval(x, {"__builtins__": {}}, env)) for x in vals]
    to = lambda t: np.array([rows[t][i] for i in sorted(rows[t])])[:, None, :]
    return to("q"), to("k"), to("v"), to("o")


def test_hand_worked_example():
    q, k, v, o = _parse_golden_attention()
    got = attend_last(q, k, v)
    np.testing.assert_allclose(got, o, rtol=0, atol=1e-13)


@pytest.mark.parametrize("L,n", [(1, 1), (5, 5), (37, 37), (37, 9), (64, 1)])
def test_zero_query_gives_running_mean(L, n):
    """Q = 0 makes every visible key equally likely: o_i = mean(V[0..p_i]) exactly."""
    rng = np.random.default_rng(L * 100 + n)
    hq, hkv, d = 4, 2, 8
    q = np.zeros((n, hq, d))
    k = rng.standard_normal((L, hkv, d))
    v = rng.standard_normal((L, hkv, d))
    got = attend_last(q, k, v)
    for i in range(n):
        p = L - n + i
        for h in range(hq):
            g = h // (hq // hkv)
            np.testing.assert_allclose(got[i, h], v[: p + 1, g].mean(axis=0), rtol=0, atol=1e-14)


def test_single_token_is_its_value():
    rng = np.random.default_rng(3)
    q, k, v = rand_case(rng, 1, 1, 4, 2, 16, scale=3.0)
    got = attend_last(q, k, v)
    for h in range(4):
        assert np.array_equal(got[0, h], v[0, h // 2])


def test_concentration_on_aligned_key():
    rng = np.random.default_rng(11)
    L, d = 30, 16
    k = rng.standard_normal((L, 1, d))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = rng.standard_normal((L, 1, d))
    for jstar in (0, 7, 29):
        q = (200.0 * k[jstar])[None]         # q . k_j* is the unique maximum by a wide margin
        got = attend_rows(q, [L - 1], k, v)
        np.testing.assert_allclose(got[0, 0], v[jstar, 0], atol=1e-8)


def brute_weights(q_row, pos, k_head):
    """Pure-Python softmax(q . k_j / sqrt(d)) over keys 0..pos, zeros after: independent of the oracle."""
    d = len(q_row)
    s = [math.fsum(q_row[e] * k_head[j][e] for e in range(d)) / math.sqrt(d) for j in range(pos + 1)]
    m = max(s)
    e = [math.exp(x - m) for x in s]
    z = math.fsum(e)
    return [x / z for x in e]


@pytest.mark.parametrize("seed", range(6))
def test_weights_match_brute_force_softmax(seed):
    """The weights attend_rows forms, scale 1/sqrt(d) included, against a brute-force softmax."""
    rng = np.random.default_rng(100 + seed)
    d = [4, 16, 64][seed % 3]
    L = int(rng.integers(1, 30))
    k = rng.standard_normal((L, d)) * 2.0
    pos = rng.integers(0, L, size=5)
    q = rng.standard_normal((5, d)) * 2.0
    w = weights(q, pos, k)
    assert w.shape == (5, int(pos.max()) + 1)
    for i in range(5):
        ref = brute_weights(q[i].tolist(), int(pos[i]), k.tolist())
        np.testing.assert_allclose(w[i, : pos[i] + 1], ref, rtol=1e-12, atol=1e-300)
        assert (w[i, pos[i] + 1:] == 0).all()                 # keys past the row are masked exactly


def test_weights_rows_scaled_far_apart():
    """A stable softmax per row: one row's scores near 0, another's in the thousands."""
    rng = np.random.default_rng(21)
    k = rng.standard_normal((6, 4)) * 3
    q = np.stack([rng.standard_normal(4), 200 * k[5]])     # second row: score 100 |k5|^2 >> 745
    w = weights(q, [5, 5], k)
    for i in range(2):
        np.testing.assert_allclose(w[i], brute_weights(q[i].tolist(), 5, k.tolist()), rtol=1e-12, atol=0)


def test_weights_hand_worked_example():
    """d = 4 (scale 1/2): q = (2 ln 2, 2 ln 3, 0, 0) against k0 = 0, k1 = e0, k2 = e1 scores
    (0, ln 2, ln 3), so the weights are (1, 2, 3) / 6 at position 2 and (1, 2) / 3 at position 1."""
    k = np.array([[0, 0, 0, 0], [1, 0, 0, 0], [0, 1, 0, 0]], dtype=np.float64)
    q = np.array([[2 * math.log(2), 2 * math.log(3), 0, 0]] * 2)
    w = weights(q, [2, 1], k)
    np.testing.assert_allclose(w, [[1 / 6, 2 / 6, 3 / 6], [1 / 3, 2 / 3, 0.0]], rtol=0, atol=1e-15)


def test_weights_rows_sum_to_one_and_give_attend_rows():
    """Every weight row of attend_rows' own softmax sums to 1, and weights @ V is its output."""
    rng = np.random.default_rng(5)
    L, hq, hkv, d = 50, 4, 2, 32
    k = rng.standard_normal((L, hkv, d)) * 4
    v = rng.standard_normal((L, hkv, d))
    q = rng.standard_normal((7, hq, d)) * 4
    pos = np.array([0, 1, 17, 49, 30, 2, 48])
    out = attend_rows(q, pos, k, v)
    for h in range(hq):
        g = kv_head_of(h, hq, hkv)
        w = weights(q[:, h], pos, k[:, g])
        assert (w >= 0).all()
        for i in range(len(pos)):
            assert abs(math.fsum(w[i]) - 1.0) <= 1e-12
        np.testing.assert_allclose(w @ v[: w.shape[1], g], out[:, h], rtol=0, atol=1e-13)


def test_gqa_equals_mha_with_repeated_kv():
    rng = np.random.default_rng(8)
    L, n, hq, hkv, d = 33, 11, 8, 2, 16
    q, k, v = rand_case(rng, L, n, hq, hkv, d)
    grp = hq // hkv
    k_rep = np.repeat(k, grp, axis=1)      # head h of the MHA copy holds KV head h // grp
    v_rep = np.repeat(v, grp, axis=1)
    a = attend_last(q, k, v)
    b = attend_last(q, k_rep, v_rep)
    np.testing.assert_allclose(a, b, rtol=0, atol=1e-14)
    assert [kv_head_of(h, hq, hkv) for h in range(hq)] == [0, 0, 0, 0, 1, 1, 1, 1]


def test_chunked_extend_equals_one_shot_prefill():
    rng = np.random.default_rng(9)
    L, hq, hkv, d = 70, 4, 2, 8
    q, k, v = rand_case(rng, L, L, hq, hkv, d)
    full = attend_last(q, k, v)
    cuts = [0, 16, 17, 40, 69, 70]
    parts = [attend_last(q[a:b], k[:b], v[:b]) for a, b in zip(cuts[:-1], cuts[1:])]
    np.testing.assert_allclose(np.concatenate(parts), full, rtol=0, atol=1e-14)


def test_decode_equals_last_prefill_row():
    rng = np.random.default_rng(10)
    L, hq, hkv, d = 45, 4, 1, 8
    q, k, v = rand_case(rng, L, L, hq, hkv, d)
    full = attend_last(q, k, v)
    dec = attend_last(q[-1:], k, v)
    np.testing.assert_allclose(dec[0], full[-1], rtol=0, atol=1e-14)


def test_empty_query_set():
    rng = np.random.default_rng(1)
    _, k, v = rand_case(rng, 5, 1, 2, 1, 4)
    assert attend_last(np.zeros((0, 2, 4)), k, v).shape == (0, 2, 4)


# ----------------------------------------------------------------------------------- wire format
def _parse_wire_golden():
    with open(os.path.join(GOLDEN, "wire_tiny.txt")) as f:
        lines = [l.split("#")[0].split() for l in f]
    lines = [l for l in lines if l]
    shape = [int(x) for x in lines[0][1:]]
    k = [int(x) for x in lines[1][1:]]
    v = [int(x) for x in lines[2][1:]]
    wire = [int(x) for l in lines[3:] for x in l[1:]]
    return shape, np.array(k), np.array(v), np.array(wire, dtype=np.uint16)


def test_wire_hand_written_golden():
    (nl, L, hkv, d), k, v, wire = _parse_wire_golden()
    kk = k.reshape(nl, L, hkv, d).astype(np.uint16)
    vv = v.reshape(nl, L, hkv, d).astype(np.uint16)
    got = kvwire.serialize(kk, vv)
    assert got.dtype == np.uint16 and got.size * 2 == kvwire.wire_bytes(nl, L, hkv, d)
    assert np.array_equal(got, wire)


def test_wire_hand_written_golden_d64_sub_blocks():
    lines = [l.split("#")[0].split() for l in open(os.path.join(GOLDEN, "wire_d64_two_tokens.txt"))]
    lines = [l for l in lines if l]
    nl, L, hkv, d = [int(x) for x in lines[0][1:]]
    want = np.zeros(kvwire.wire_bytes(nl, L, hkv, d) // 2, dtype=np.uint16)
    for l in lines[1:]:
        assert l[0] == "runs"
        P, N, V, S, R, PS, VS = (int(x) for x in l[1:])
        for r in range(R):
            for i in range(N):
                want[P + r * PS + i] = V + r * VS + i * S
    t = np.arange(L)[:, None]
    j = np.arange(d)[None, :]
    k = (1000 + 100 * t + j).astype(np.uint16).reshape(nl, L, hkv, d)
    v = (5000 + 100 * t + j).astype(np.uint16).reshape(nl, L, hkv, d)
    assert np.array_equal(kvwire.serialize(k, v), want)
    k2, v2 = kvwire.deserialize(want, nl, L, hkv, d)
    assert np.array_equal(k2, k) and np.array_equal(v2, v)


@pytest.mark.parametrize("d", [8, 64])
@pytest.mark.parametrize("L", [1, 15, 16, 17, 48, 100])
def test_wire_round_trip_and_zero_tail(L, d):
    rng = np.random.default_rng(L)
    nl, hkv = 2, 3
    k = rng.integers(1, 65536, size=(nl, L, hkv, d), dtype=np.uint16)
    v = rng.integers(1, 65536, size=(nl, L, hkv, d), dtype=np.uint16)
    w = kvwire.serialize(k, v)
    assert w.size * 2 == kvwire.wire_bytes(nl, L, hkv, d)
    k2, v2 = kvwire.deserialize(w, nl, L, hkv, d)
    assert np.array_equal(k, k2) and np.array_equal(v, v2)
    assert np.array_equal(kvwire.serialize(k2, v2), w)
    pages = (L + 15) // 16
    blk = w.reshape(nl, pages, hkv, 2, 16 * d)
    tail = L - (pages - 1) * 16
    sw = min(d, 32)                                        # K sub-blocks [d/sw][16][sw]
    kl = blk[:, -1, :, 0].reshape(nl, hkv, d // sw, 16, sw).transpose(0, 1, 3, 2, 4)
    vl = blk[:, -1, :, 1].reshape(nl, hkv, d, 16)
    assert (kl[:, :, tail:] == 0).all() and (vl[:, :, :, tail:] == 0).all()
    # every nonzero input value appears exactly once in the wire (pure movement)
    assert np.count_nonzero(w) == 2 * k.size


def test_conversation_store_is_concatenation():
    c = kvwire.ConversationKV(2, 1, 4)
    a = np.arange(2 * 3 * 4, dtype=np.uint16).reshape(2, 3, 1, 4)
    b = (100 + np.arange(2 * 2 * 4, dtype=np.uint16)).reshape(2, 2, 1, 4)
    c.append(a, a + 1)
    c.append(b, b + 1)
    assert c.length == 5
    assert np.array_equal(c.k[:, :3], a) and np.array_equal(c.k[:, 3:], b)
    assert np.array_equal(c.v[:, 3:], b + 1)
