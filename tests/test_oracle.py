"""Pins for the fp64 oracle (CPU only).

Each check ties the oracle to something other than itself: a brute-force
dense-mask computation built from logical arrays (never from the pool), a
library softmax / logsumexp, torch's causal SDPA, closed forms, invariants,
and a hand-solved example.  Several tests plant plausible mistakes in a copy
of the oracle and check that the pins catch them.
"""

import math
import os

import numpy as np
import pytest
import scipy.special as sps

import oracle
from oracle import attention as OA
from paper_2608_25523_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- helpers

def _bits(x):
    """float -> bf16 bits; the test only uses values exact in bf16."""
    b = W.bf16_round(np.asarray(x, np.float32))
    assert np.array_equal(OA.bf16_bits_to_f64(b), np.asarray(x, np.float64)), "value not exact in bf16"
    return b


def _random_bf16_values(rng, shape, scale=1.0):
    return OA.bf16_bits_to_f64(W.bf16_round((rng.standard_normal(shape) * scale).astype(np.float32)))


class Tiny:
    """A small batch built from logical arrays, then scattered into a pool."""

    def __init__(self, seed, hq=4, hkv=2, d=8, prefix=(5, 19), reqs=((0, 7, 7), (1, 20, 1), (-1, 9, 9), (1, 33, 3), (0, 16, 16)),
                 num_pages=64, values=None):
        rng = np.random.default_rng(seed)
        self.hq, self.hkv, self.d = hq, hkv, d
        self.prefix_len = np.array(prefix, np.int32)
        self.agent = np.array([r[0] for r in reqs], np.int32)
        self.suffix_len = np.array([r[1] for r in reqs], np.int32)
        self.n_rows = np.array([r[2] for r in reqs], np.int32)
        gen = values or (lambda shape: _random_bf16_values(rng, shape))
        self.kpre = [gen((p, hkv, d)) for p in prefix]
        self.vpre = [gen((p, hkv, d)) for p in prefix]
        self.ksuf = [gen((l, hkv, d)) for l in self.suffix_len]
        self.vsuf = [gen((l, hkv, d)) for l in self.suffix_len]
        self.q = gen((int(self.n_rows.sum()), hq, d))
        self.num_pages = num_pages
        self.place(rng)

    def place(self, rng):
        perm = rng.permutation(self.num_pages)
        at = 0
        pool_k = np.full((self.num_pages, self.hkv, 16, self.d), W.POISON_BF16, np.uint16)
        pool_v = pool_k.copy()
        self.prefix_pages, self.suffix_pages = [], []

        def put(k, v):
            nonlocal at
            pages = []
            for j in range(k.shape[0]):
                if j % 16 == 0:
                    pages.append(int(perm[at]))
                    at += 1
                pool_k[pages[-1], :, j % 16, :] = _bits(k[j])
                pool_v[pages[-1], :, j % 16, :] = _bits(v[j])
            return np.array(pages, np.int32)

        for k, v in zip(self.kpre, self.vpre):
            self.prefix_pages.append(put(k, v))
        for k, v in zip(self.ksuf, self.vsuf):
            self.suffix_pages.append(put(k, v))
        self.pool_k, self.pool_v = pool_k, pool_v
        self.q_bits = _bits(self.q)

    def oracle(self, fn=None, **kw):
        fn = fn or oracle.prefix_shared_attention
        return fn(self.pool_k, self.pool_v, self.prefix_pages, self.prefix_len, self.agent,
                  self.suffix_pages, self.suffix_len, self.n_rows, self.q_bits, self.hq, **kw)

    def brute_force(self, scale=None):
        """Dense-mask attention over the concatenated logical sequence using
        scipy's softmax and logsumexp; never touches the pool."""
        scale = 1.0 / math.sqrt(self.d) if scale is None else scale
        kv_of_head = np.repeat(np.arange(self.hkv), self.hq // self.hkv)
        o = np.zeros((self.q.shape[0], self.hq, self.d))
        lse = np.zeros((self.q.shape[0], self.hq))
        row = 0
        for r in range(len(self.agent)):
            a = self.agent[r]
            kseq = self.ksuf[r] if a < 0 else np.concatenate([self.kpre[a], self.ksuf[r]])
            vseq = self.vsuf[r] if a < 0 else np.concatenate([self.vpre[a], self.vsuf[r]])
            total = kseq.shape[0]
            n = self.n_rows[r]
            mask = np.zeros((n, total), bool)
            for i in range(n):
                mask[i, : total - n + i + 1] = True
            for h in range(self.hq):
                s = np.einsum("id,jd->ij", self.q[row:row + n, h], kseq[:, kv_of_head[h]]) * scale
                s = np.where(mask, s, -np.inf)
                o[row:row + n, h] = sps.softmax(s, axis=1) @ vseq[:, kv_of_head[h]]
                lse[row:row + n, h] = sps.logsumexp(s, axis=1)
            row += n
        return o, lse


# ---------------------------------------------------------------- widening

def test_bf16_widening_known_patterns():
    pats = np.array([0x3F80, 0xC000, 0x4049, 0x0001, 0x7F80, 0xFF80, 0x0000, 0x8000, 0x7F7F], np.uint16)
    want = [1.0, -2.0, 3.140625, 2.0 ** -133, np.inf, -np.inf, 0.0, -0.0, 3.3895313892515355e38]
    got = OA.bf16_bits_to_f64(pats)
    assert got.dtype == np.float64
    np.testing.assert_array_equal(got, want)
    assert np.isnan(OA.bf16_bits_to_f64(np.array([W.POISON_BF16], np.uint16)))[0]


def test_bf16_round_ties_to_even():
    # 1 + 2^-8 lies halfway between bf16 1.0 and 1 + 2^-7: rounds to even (1.0)
    x = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -1 - 2 ** -8, 1 + 2 ** -8 + 2 ** -20], np.float32)
    np.testing.assert_array_equal(W.bf16_round(x), np.array([0x3F80, 0x3F82, 0xBF80, 0x3F81], np.uint16))


# ---------------------------------------------------------------- brute force

@pytest.mark.parametrize("seed", [0, 1, 2])
def test_matches_brute_force_dense_mask(seed):
    t = Tiny(seed)
    o, lse = t.oracle()
    bo, bl = t.brute_force()
    assert np.max(np.abs(o - bo)) <= 1e-12
    assert np.max(np.abs(lse - bl)) <= 1e-12


def test_brute_force_gqa_group_of_four_and_custom_scale():
    t = Tiny(7, hq=8, hkv=2, d=16, prefix=(40,), reqs=((0, 18, 18), (0, 50, 1), (-1, 3, 2)))
    o, lse = t.oracle(scale=0.3)
    bo, bl = t.brute_force(scale=0.3)
    assert np.max(np.abs(o - bo)) <= 1e-12 and np.max(np.abs(lse - bl)) <= 1e-12


def test_rows_sum_to_one():
    """With V_j = e_j the output row is the softmax row itself."""
    d = 64
    rng = np.random.default_rng(3)

    def gen(shape):
        return _random_bf16_values(rng, shape)

    t = Tiny(3, hq=2, hkv=1, d=d, prefix=(20,), reqs=((0, 30, 30), (0, 12, 1)), values=gen)
    eye = np.eye(d)
    t.vpre = [eye[:20, None, :]]
    t.vsuf = [eye[20:50, None, :], eye[20:32, None, :]]
    t.place(np.random.default_rng(4))
    o, _ = t.oracle()
    sums = o.sum(axis=2)
    assert np.max(np.abs(sums - 1.0)) <= 1e-12
    assert np.all(o >= 0)
    # each row puts weight only on the keys it may see
    row = 0
    for i in range(30):
        assert np.all(o[row + i, :, 20 + i + 1:] == 0)
    bo, _ = t.brute_force()
    assert np.max(np.abs(o - bo)) <= 1e-12


# ---------------------------------------------------------------- split / merge

@pytest.mark.parametrize("seed", [0, 5, 11])
def test_split_merge_equals_monolithic(seed):
    t = Tiny(seed)
    o, lse = t.oracle()
    rng = np.random.default_rng(seed + 100)
    for pc, sc in [(None, None), (4, None), (None, 3), (7, 5), (1, 1)]:
        so, sl = t.oracle(OA.split_attention, prefix_chunk=pc, suffix_chunk=sc, rng=rng)
        assert np.max(np.abs(so - o)) <= 1e-12
        assert np.max(np.abs(sl - lse)) <= 1e-12


def test_merge_partials_closed_form():
    # two halves with equal LSE combine to the average and gain ln 2
    o1, o2 = np.array([1.0, 3.0]), np.array([3.0, 5.0])
    o, l = oracle.merge_partials([o1, o2], [np.array(2.5), np.array(2.5)])
    np.testing.assert_allclose(o, [2.0, 4.0], atol=1e-15)
    np.testing.assert_allclose(l, 2.5 + math.log(2), atol=1e-15)
    # order does not matter, weights follow exp(lse)
    o, l = oracle.merge_partials([o2, o1], [np.array(0.0), np.array(math.log(3))])
    np.testing.assert_allclose(o, 0.25 * o2 + 0.75 * o1, atol=1e-15)
    np.testing.assert_allclose(l, math.log(4), atol=1e-15)


# ---------------------------------------------------------------- closed forms

def test_zero_query_gives_mean_of_visible_values():
    t = Tiny(9)
    t.q = np.zeros_like(t.q)
    t.q_bits = _bits(t.q)
    o, lse = t.oracle()
    row = 0
    for r in range(len(t.agent)):
        a = t.agent[r]
        vseq = t.vsuf[r] if a < 0 else np.concatenate([t.vpre[a], t.vsuf[r]])
        n = t.n_rows[r]
        for i in range(n):
            pos = vseq.shape[0] - n + i
            mean = vseq[: pos + 1].mean(axis=0)           # [Hkv][d]
            for h in range(t.hq):
                np.testing.assert_allclose(o[row + i, h], mean[h // (t.hq // t.hkv)], atol=1e-13)
                assert abs(lse[row + i, h] - math.log(pos + 1)) <= 1e-13
        row += n


def test_constant_values_reproduced():
    t = Tiny(10)
    c = 1.5
    t.vpre = [np.full_like(v, c) for v in t.vpre]
    t.vsuf = [np.full_like(v, c) for v in t.vsuf]
    t.place(np.random.default_rng(1))
    o, _ = t.oracle()
    assert np.max(np.abs(o - c)) <= 1e-13


def test_one_hot_query_selects_value_row():
    d, plen, slen = 32, 12, 10
    rng = np.random.default_rng(12)

    def gen(shape):
        return _random_bf16_values(rng, shape)

    t = Tiny(12, hq=1, hkv=1, d=d, prefix=(plen,), reqs=((0, slen, 1),), values=gen)
    eye = np.eye(d)
    t.kpre = [eye[:plen, None, :]]
    t.ksuf = [eye[plen:plen + slen, None, :]]
    for jstar in [0, 5, plen + 3, plen + slen - 1]:
        t.q = (512.0 * eye[jstar])[None, None, :]
        t.place(np.random.default_rng(jstar))
        o, lse = t.oracle()
        vseq = np.concatenate([t.vpre[0], t.vsuf[0]])[:, 0]
        np.testing.assert_allclose(o[0, 0], vseq[jstar], atol=1e-9)
        assert abs(lse[0, 0] - 512.0 / math.sqrt(d)) < 1e-9


def test_no_prefix_equals_torch_causal_sdpa():
    torch = pytest.importorskip("torch")
    t = Tiny(13, hq=4, hkv=4, d=16, prefix=(), reqs=((-1, 37, 37),))
    o, _ = t.oracle()
    q = torch.tensor(t.q).permute(1, 0, 2)[None]                  # [1][H][n][d]
    k = torch.tensor(t.ksuf[0]).permute(1, 0, 2)[None]
    v = torch.tensor(t.vsuf[0]).permute(1, 0, 2)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True)
    ref = ref[0].permute(1, 0, 2).numpy()
    assert np.max(np.abs(o - ref)) <= 1e-12


def test_two_key_hand_example():
    vals = {}
    with open(os.path.join(GOLDEN, "two_key_closed_form.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                name, *xs = line.split()
                vals[name] = np.array([float(x) for x in xs])
    pool = np.zeros((3, 1, 16, 2), np.uint16)
    pool_v = pool.copy()
    pool[0, 0, 0], pool_v[0, 0, 0] = _bits(vals["k0"]), _bits(vals["v0"])   # prefix page
    pool[1, 0, 0], pool_v[1, 0, 0] = _bits(vals["k1"]), _bits(vals["v1"])   # suffix of request 0
    pool[2, 0, 0], pool_v[2, 0, 0] = _bits(vals["k1"]), _bits(vals["v1"])   # suffix of request 1
    q = _bits(np.stack([vals["q_row0"], vals["q_row1"]])[:, None, :])
    o, lse = oracle.prefix_shared_attention(pool, pool_v, [np.array([0])], [1], [0, 0],
                                            [np.array([1]), np.array([2])], [1, 1], [1, 1], q, 1)
    e = math.exp(math.sqrt(2))
    np.testing.assert_allclose(o[0, 0], [1 / (1 + e), e / (1 + e)], atol=1e-15)
    assert abs(lse[0, 0] - math.log(1 + e)) < 1e-15
    np.testing.assert_allclose(o[1, 0], [0.5, 0.5], atol=1e-15)
    assert abs(lse[1, 0] - math.log(2)) < 1e-15


# ---------------------------------------------------------------- structure invariants

def test_decode_row_equals_extend_row():
    t = Tiny(14, prefix=(21,), reqs=((0, 40, 40),))
    ext_o, ext_l = t.oracle()
    for pos in [0, 1, 15, 16, 39]:
        o, l = oracle.prefix_shared_attention(t.pool_k, t.pool_v, t.prefix_pages, t.prefix_len, t.agent,
                                              t.suffix_pages, np.array([pos + 1]), np.array([1]),
                                              t.q_bits[pos:pos + 1], t.hq)
        # same arithmetic up to BLAS summation order
        np.testing.assert_allclose(o[0], ext_o[pos], rtol=0, atol=1e-14)
        np.testing.assert_allclose(l[0], ext_l[pos], rtol=0, atol=1e-14)


def test_page_placement_invariance():
    t = Tiny(15)
    o1, l1 = t.oracle()
    t.place(np.random.default_rng(99))
    o2, l2 = t.oracle()
    np.testing.assert_array_equal(o1, o2)
    np.testing.assert_array_equal(l1, l2)


def test_row_subset_matches_full():
    t = Tiny(16)
    o, l = t.oracle()
    sub = {0: [0, 6], 3: [2], 4: [15]}
    so, sl = t.oracle(rows=sub)
    offs = np.concatenate([[0], np.cumsum(t.n_rows)])
    for r, rows in sub.items():
        for i in rows:
            np.testing.assert_allclose(so[offs[r] + i], o[offs[r] + i], rtol=0, atol=1e-14)
    assert np.isnan(so[offs[1]]).all()


# ---------------------------------------------------------------- byte movement

def test_append_kv_writes_suffix_tail_only():
    rng = np.random.default_rng(17)
    pool_k = rng.integers(0, 65535, size=(10, 2, 16, 4), dtype=np.uint16)
    pool_v = rng.integers(0, 65535, size=(10, 2, 16, 4), dtype=np.uint16)
    suffix_pages = [np.array([3, 7]), np.array([1])]
    suffix_len, n_rows = [20, 5], [3, 5]
    kn = rng.integers(0, 65535, size=(8, 2, 4), dtype=np.uint16)
    vn = rng.integers(0, 65535, size=(8, 2, 4), dtype=np.uint16)
    ok, ov = oracle.append_kv(pool_k, pool_v, suffix_pages, suffix_len, n_rows, kn, vn)
    want_k = pool_k.copy()
    want_k[7, :, 1] = kn[0]; want_k[7, :, 2] = kn[1]; want_k[7, :, 3] = kn[2]   # positions 17, 18, 19
    for i in range(5):
        want_k[1, :, i] = kn[3 + i]                                                  # positions 0..4
    np.testing.assert_array_equal(ok, want_k)
    assert np.array_equal(ov[7, :, 3], vn[2]) and np.array_equal(ov[1, :, 4], vn[7])
    changed = np.argwhere(np.any(ok != pool_k, axis=(1, 3)))
    assert {tuple(x) for x in changed} <= {(7, 1), (7, 2), (7, 3), (1, 0), (1, 1), (1, 2), (1, 3), (1, 4)}


def test_page_copy_bytes():
    rng = np.random.default_rng(18)
    src = rng.integers(0, 65535, size=(5, 2, 16, 4), dtype=np.uint16)
    dst = rng.integers(0, 65535, size=(9, 2, 16, 4), dtype=np.uint16)
    out = oracle.page_copy(dst, src, [8, 0, 4], [1, 4, 1])
    np.testing.assert_array_equal(out[8], src[1])
    np.testing.assert_array_equal(out[0], src[4])
    np.testing.assert_array_equal(out[4], src[1])
    for p in [1, 2, 3, 5, 6, 7]:
        np.testing.assert_array_equal(out[p], dst[p])


# ---------------------------------------------------------------- the pins catch planted mistakes

def _mutant(monkeypatch, which):
    """Plant a plausible mistake in the oracle (CPU only) and return it."""
    orig = OA.attend_rows

    def wrong(q, k, v, positions, num_q_heads, scale, heads=None):
        if which == "off_by_one_mask":
            positions = [p - 1 if p > 0 else p for p in positions]
        elif which == "gqa_modulo":
            hkv = k.shape[1]
            k = k[:, [(h % hkv) for h in range(hkv)][::-1], :] if hkv > 1 else k
        elif which == "no_scale":
            scale = 1.0
        elif which == "transposed_pv":
            v = v[::-1]
        return orig(q, k, v, positions, num_q_heads, scale, heads)

    monkeypatch.setattr(OA, "attend_rows", wrong)


@pytest.mark.parametrize("which", ["off_by_one_mask", "gqa_modulo", "no_scale", "transposed_pv"])
def test_brute_force_catches_planted_mistakes(monkeypatch, which):
    t = Tiny(21)
    bo, bl = t.brute_force()
    _mutant(monkeypatch, which)
    o, l = t.oracle()
    assert max(np.max(np.abs(o - bo)), np.max(np.abs(l - bl))) > 1e-6


def test_merge_pin_catches_wrong_merge(monkeypatch):
    t = Tiny(22)
    o, _ = t.oracle()

    def bad_merge(o_parts, lse_parts):
        lse = np.log(sum(np.exp(l) for l in lse_parts))
        return sum(o_parts) / len(o_parts), lse                # forgets the weights

    monkeypatch.setattr(OA, "merge_partials", bad_merge)
    so, _ = t.oracle(OA.split_attention, prefix_chunk=4, suffix_chunk=3)
    assert np.max(np.abs(so - o)) > 1e-6
