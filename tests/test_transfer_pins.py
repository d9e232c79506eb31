"""Pins of the transfer oracle (Sec. 6.1 CPU-assisted prefetch; Sec. 6.2
Copy-out / Copy-in; App. A.3 record sizes; App. A.4 fp32 gradients).

Independent formulations only: a record packed by hand with ``struct``,
round trips through copy_out and copy_in, an fp32 case whose result depends
on the order of the additions (worked out by hand), sums of exactly
representable integers, the fp32 rounding bound against an fp64 sum, and
brute-force properties of the prefetch plan. Mutation tests plant plausible
mistakes in the oracle (on the CPU) and require a pin to catch them.
"""
import struct

import numpy as np
import pytest

import oracle.foremoe_transfer as X


def _arrays(W, G, d, F, rng, p_dtype=np.uint16):
    if p_dtype == np.uint16:
        wgu = rng.integers(0, 1 << 16, size=(W, 2 * F, d)).astype(np.uint16)
        wdn = rng.integers(0, 1 << 16, size=(W, d, F)).astype(np.uint16)
    else:
        wgu = rng.standard_normal((W, 2 * F, d)).astype(np.float32)
        wdn = rng.standard_normal((W, d, F)).astype(np.float32)
    ggu = rng.standard_normal((G, 2 * F, d)).astype(np.float32)
    gdn = rng.standard_normal((G, d, F)).astype(np.float32)
    return wgu, wdn, ggu, gdn


# ---------------------------------------------------------------------------
# Record layout (Copy-out)
# ---------------------------------------------------------------------------
def check_layout_by_hand():
    # d = 2, F = 1: gate/up [2, 2] bf16, down [2, 1] bf16, then the fp32
    # gradients of the same shapes: 8 + 4 + 16 + 8 = 36 bytes = 3*d*F*(2+4)
    wgu = np.zeros((2, 2, 2), np.uint16)
    wdn = np.zeros((2, 2, 1), np.uint16)
    wgu[1] = [[1, 2], [3, 4]]
    wdn[1] = [[5], [6]]
    ggu = np.zeros((2, 2, 2), np.float32)
    gdn = np.zeros((2, 2, 1), np.float32)
    ggu[0] = [[1.0, 2.0], [3.0, 4.0]]
    gdn[0] = [[5.0], [6.0]]
    rec = struct.pack("<4H2H4f2f", 1, 2, 3, 4, 5, 6, 1.0, 2.0, 3.0, 4.0, 5.0, 6.0)
    both = X.copy_out(wgu, wdn, ggu, gdn, [1], [0], X.PARAMS | X.GRADS).tobytes() == rec
    # two records, parameters only: record i at offset 12 i
    two = X.copy_out(wgu, wdn, ggu, gdn, [1, 0], [0, 0], X.PARAMS).tobytes() == \
        struct.pack("<6H6H", 1, 2, 3, 4, 5, 6, 0, 0, 0, 0, 0, 0)
    grads = X.copy_out(wgu, wdn, ggu, gdn, [0], [0], X.GRADS).tobytes() == rec[12:]
    return both and two and grads and X.record_bytes(2, 1, 2, X.PARAMS | X.GRADS) == 36


def test_layout_by_hand():
    assert check_layout_by_hand()


def test_record_bytes_app_a():
    # App. A.4: Qwen3-30B-A3B, h = 2048, h_ff = 768, bf16 weights and fp32
    # gradients: S_e = 9.0 MiB, S_g = 18.0 MiB per expert
    assert X.record_bytes(2048, 768, 2, X.PARAMS) == 9 * 2 ** 20
    assert X.record_bytes(2048, 768, 2, X.GRADS) == 18 * 2 ** 20
    assert X.record_bytes(2048, 768, 2, X.PARAMS | X.GRADS) == 27 * 2 ** 20


@pytest.mark.parametrize("p_dtype", [np.uint16, np.float32])
def test_round_trip_moves_experts(p_dtype):
    # experts leave weight/gradient slots a and land in slots b of another
    # GPU's arrays: exactly their bytes arrive, nothing else changes
    rng = np.random.default_rng(1)
    d, F = 8, 4
    src = _arrays(5, 5, d, F, rng, p_dtype)
    dst = _arrays(6, 6, d, F, rng, p_dtype)
    a, b = [4, 0, 2], [1, 5, 3]
    buf = X.copy_out(*src, a, a, X.PARAMS | X.GRADS)
    assert buf.size == 3 * X.record_bytes(d, F, np.dtype(p_dtype).itemsize, X.PARAMS | X.GRADS)
    out = X.copy_in(buf, b, b, [X.ASSIGN] * 3, X.PARAMS | X.GRADS, *dst)
    for o, s, t in zip(out, src, dst):
        for i, j in zip(a, b):
            assert np.array_equal(o[j].view(np.uint8), np.ascontiguousarray(s[i]).view(np.uint8))
        for j in set(range(t.shape[0])) - set(b):
            assert np.array_equal(o[j].view(np.uint8), t[j].view(np.uint8))


def test_copy_in_skips_negative_targets():
    rng = np.random.default_rng(2)
    src = _arrays(2, 2, 4, 2, rng)
    dst = _arrays(3, 3, 4, 2, rng)
    buf = X.copy_out(*src, [0, 1], [0, 1], X.PARAMS | X.GRADS)
    out = X.copy_in(buf, [-1, 2], [1, -1], [X.ASSIGN, X.ASSIGN], X.PARAMS | X.GRADS, *dst)
    assert np.array_equal(out[0][2], src[0][1]) and np.array_equal(out[0][:2], dst[0][:2])
    assert np.array_equal(out[2][1], src[2][0]) and np.array_equal(out[2][[0, 2]], dst[2][[0, 2]])


# ---------------------------------------------------------------------------
# Main-expert gradient accumulation (Copy-in)
# ---------------------------------------------------------------------------
def check_accumulation_order():
    # fp32 keeps 24 significant bits. Target 0 starts at 0; three replica
    # partial gradients 2^24, 1, 1 are added in record order:
    # 0 + 2^24 = 2^24; 2^24 + 1 = 16777217 is a tie between 2^24 and
    # 2^24 + 2 and rounds to the even 2^24; again 2^24. (In the reverse
    # order, 1 + 1 = 2 and 2 + 2^24 = 16777218 exactly.)
    d, F = 1, 1
    def z(G):
        return np.zeros((G, 2 * F, d), np.float32), np.zeros((G, d, F), np.float32)

    src_gu, src_dn = z(3)
    for i, v in enumerate([2.0 ** 24, 1.0, 1.0]):
        src_gu[i] = v
        src_dn[i] = v
    wz = np.zeros((3, 2, 1), np.uint16), np.zeros((3, 1, 1), np.uint16)
    buf = X.copy_out(*wz, src_gu, src_dn, [0, 1, 2], [0, 1, 2], X.GRADS)
    dgu, ddn = z(1)
    out = X.copy_in(buf, [-1] * 3, [0, 0, 0], [X.ADD] * 3, X.GRADS, np.zeros((1, 2, 1), np.uint16),
                    np.zeros((1, 1, 1), np.uint16), dgu, ddn)
    return float(out[2][0, 0, 0]) == 16777216.0 and float(out[3][0, 0, 0]) == 16777216.0


def test_accumulation_order_by_hand():
    assert check_accumulation_order()


def check_integer_sums(seed=3):
    # integers below 2^20 are exact in fp32 and so are their sums here: the
    # result is the plain sum whatever the order; ASSIGN discards what the
    # target held before it
    rng = np.random.default_rng(seed)
    d, F, G = 8, 4, 3
    w0 = np.zeros((6, 2 * F, d), np.uint16), np.zeros((6, d, F), np.uint16)
    sgu = rng.integers(-1000, 1000, size=(6, 2 * F, d)).astype(np.float32)
    sdn = rng.integers(-1000, 1000, size=(6, d, F)).astype(np.float32)
    tgu = rng.integers(-1000, 1000, size=(G, 2 * F, d)).astype(np.float32)
    tdn = rng.integers(-1000, 1000, size=(G, d, F)).astype(np.float32)
    gidx = [2, 0, 2, 1, 2, 0]
    gmode = [X.ADD, X.ADD, X.ASSIGN, X.ADD, X.ADD, X.ADD]
    buf = X.copy_out(*w0, sgu, sdn, list(range(6)), list(range(6)), X.GRADS)
    out = X.copy_in(buf, [-1] * 6, gidx, gmode, X.GRADS, np.zeros((G, 2 * F, d), np.uint16),
                    np.zeros((G, d, F), np.uint16), tgu, tdn)
    exp_gu = [tgu[0] + sgu[1] + sgu[5], tgu[1] + sgu[3], sgu[2] + sgu[4]]
    exp_dn = [tdn[0] + sdn[1] + sdn[5], tdn[1] + sdn[3], sdn[2] + sdn[4]]
    return all(np.array_equal(out[2][g], exp_gu[g]) and np.array_equal(out[3][g], exp_dn[g]) for g in range(G))


def test_integer_sums():
    assert check_integer_sums()


def test_fp32_sum_within_rounding_bound_of_fp64():
    # n additions in fp32: |fl(sum) - sum| <= n * 2^-24 * sum |terms|
    rng = np.random.default_rng(4)
    d, F, n = 16, 8, 7
    w0 = np.zeros((n, 2 * F, d), np.uint16), np.zeros((n, d, F), np.uint16)
    sgu = (rng.standard_normal((n, 2 * F, d)) * 10.0 ** rng.integers(-3, 4, size=(n, 1, 1))).astype(np.float32)
    sdn = rng.standard_normal((n, d, F)).astype(np.float32)
    tgu = rng.standard_normal((1, 2 * F, d)).astype(np.float32)
    tdn = rng.standard_normal((1, d, F)).astype(np.float32)
    buf = X.copy_out(*w0, sgu, sdn, list(range(n)), list(range(n)), X.GRADS)
    out = X.copy_in(buf, [-1] * n, [0] * n, [X.ADD] * n, X.GRADS, np.zeros((1, 2 * F, d), np.uint16),
                    np.zeros((1, d, F), np.uint16), tgu, tdn)
    for got, t, s in ((out[2][0], tgu[0], sgu), (out[3][0], tdn[0], sdn)):
        exact = t.astype(np.float64) + s.astype(np.float64).sum(axis=0)
        mag = np.abs(t).astype(np.float64) + np.abs(s).astype(np.float64).sum(axis=0)
        assert np.all(np.abs(got - exact) <= n * 2.0 ** -24 * mag)


# ---------------------------------------------------------------------------
# CPU-assisted prefetch plan (Sec. 6.1)
# ---------------------------------------------------------------------------
def check_prefetch_by_hand():
    # slots hold experts 3, 7, (empty), 5; the next micro-step needs 5, 2, 3, 9.
    # 5 and 3 stay in slots 3 and 0; slots 1 (7 is not needed) and 2 (empty)
    # are free, in ascending order: 2 -> slot 1, 9 -> slot 2.
    slot_of, fetches = X.plan_prefetch([3, 7, -1, 5], [5, 2, 3, 9])
    return slot_of == [3, 1, 0, 2] and fetches == [(2, 1), (9, 2)]


def test_prefetch_by_hand():
    assert check_prefetch_by_hand()


@pytest.mark.parametrize("seed", range(4))
def test_prefetch_properties(seed):
    rng = np.random.default_rng(seed)
    for _ in range(50):
        W, E = int(rng.integers(1, 12)), 20
        resident = [int(e) if rng.random() < 0.8 else -1 for e in rng.integers(0, E, size=W)]
        needed = [int(e) for e in rng.permutation(E)[:int(rng.integers(0, W + 1))]]
        slot_of, fetches = X.plan_prefetch(resident, needed)
        # the fewest possible fetches: exactly the needed experts not resident
        assert len(fetches) == len(set(needed) - set(resident))
        after = list(resident)
        for e, w in fetches:
            after[w] = e
        assert len(set(slot_of)) == len(needed)
        assert all(after[w] == e for w, e in zip(slot_of, needed))
        # a needed expert that was resident was not moved or overwritten
        for e in set(needed) & {r for r in resident if r >= 0}:
            assert resident[slot_of[needed.index(e)]] == e


def test_prefetch_errors():
    with pytest.raises(ValueError):
        X.plan_prefetch([0, 1], [2, 3, 4])
    with pytest.raises(ValueError):
        X.plan_prefetch([0, 1], [2, 2])


# ---------------------------------------------------------------------------
# Mutation tests
# ---------------------------------------------------------------------------
def test_mutation_gradients_before_parameters_is_caught(monkeypatch):
    real = X.copy_out

    def wrong(wgu, wdn, ggu, gdn, widx, gidx, what):
        if what != X.PARAMS | X.GRADS:
            return real(wgu, wdn, ggu, gdn, widx, gidx, what)
        parts = []
        for i in range(len(widx)):
            parts.append(real(wgu, wdn, ggu, gdn, [widx[i]], [gidx[i]], X.GRADS))
            parts.append(real(wgu, wdn, ggu, gdn, [widx[i]], [gidx[i]], X.PARAMS))
        return np.concatenate(parts)

    monkeypatch.setattr(X, "copy_out", wrong)
    assert not check_layout_by_hand()


def test_mutation_reverse_accumulation_order_is_caught(monkeypatch):
    real = X.copy_in

    def wrong(buf, widx, gidx, gmode, what, *arrs):
        W, F2, d = arrs[0].shape
        rb = X.record_bytes(d, F2 // 2, arrs[0].dtype.itemsize, what)
        n = len(widx)
        rev = np.concatenate([buf[i * rb:(i + 1) * rb] for i in reversed(range(n))]) if n else buf
        return real(rev, widx[::-1], gidx[::-1], gmode[::-1], what, *arrs)

    monkeypatch.setattr(X, "copy_in", wrong)
    assert not check_accumulation_order()


def test_mutation_add_as_assign_is_caught(monkeypatch):
    real = X.copy_in
    monkeypatch.setattr(X, "copy_in", lambda buf, widx, gidx, gmode, what, *a:
                        real(buf, widx, gidx, [X.ASSIGN] * len(gmode), what, *a))
    assert not check_integer_sums()


def test_mutation_prefetch_refetches_resident_is_caught(monkeypatch):
    real = X.plan_prefetch
    monkeypatch.setattr(X, "plan_prefetch", lambda resident, needed: real([-1] * len(resident), needed))
    assert not check_prefetch_by_hand()
