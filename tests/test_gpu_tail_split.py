"""Row GEMMs, the partial last round of output tiles: with 256-wide tiles
a round of at most 7/16 of the workgroups is cut along N into half-width
tiles, and with the optional workspace each (half) tile of a long enough
GEMM is cut along K into up to 4 pieces whose fp32 partial sums the last
piece to finish adds in piece order (grouped SwiGLU FFN of App. A; the cuts
only change where and in which fp32 order the Step-4 products are summed).

Row layouts are chosen so that the cuts really happen (the expected layout
per GEMM is computed here from the tile counts and asserted on 256 CUs):
halves alone, halves in 2, 3 and 4 K pieces, 128-wide tiles (F not a
multiple of 256) in 2, 3 and 4 K pieces, and no cut. Checked: sampled rows
or every row against the fp64 oracle, with against without workspace within
the tolerance, two runs bit for bit equal, and the arrival counters left at
zero.
"""
import numpy as np
import pytest
import torch

import oracle.foremoe_oracle as O
from gpu_helpers import check_close, to_np
from workload import bf16_round

pytestmark = pytest.mark.gpu

D, W = 2048, 3
SPLIT_MAX, SPLIT_MIN_K = 4, 32


def expected_layout(rows, n_cols, k, grid, with_ws=True):
    """(halves, pieces) of the last round's tiles, as the kernel picks them:
    256-wide output tiles when n_cols allows (else 128-wide); a partial last
    round of at most 7/16 of the workgroups is cut along N into two
    half-width tiles (256-wide tiles only); then, with a workspace and at
    least SPLIT_MIN_K k-steps, each (half) tile along K into as many pieces
    as keep at most 7/8 of the workgroups busy, at most SPLIT_MAX."""
    bn = 256 if n_cols % 256 == 0 else 128
    tiles = sum((r + 255) // 256 for r in rows) * (n_cols // bn)
    rem = tiles % grid
    if rem == 0:
        return 1, 1
    halves = 2 if bn == 256 and 16 * rem <= 7 * grid else 1
    pieces = 1
    if with_ws and k // 64 >= SPLIT_MIN_K:
        pieces = min((7 * grid // 8) // (rem * halves), SPLIT_MAX)
        pieces = pieces if pieces >= 2 else 1
    return halves, pieces


def sampled(off, rng, per_slot=5):
    rows, sub, widx = [], [0], []
    for j in range(len(off) - 1):
        lo, hi = int(off[j]), int(off[j + 1])
        if hi <= lo:
            continue
        pick = np.unique(np.concatenate([[lo, hi - 1], rng.integers(lo, hi, size=per_slot)]))
        rows.extend(pick.tolist())
        sub.append(sub[-1] + len(pick))
        widx.append(j % W)
    return np.array(rows), np.array(sub), np.array(widx)


# (F, rows of each slot, expected (halves, pieces) of the gate/up forward
# and of the down dgrad on a 256-CU MI355X, both with K = d = 2048): 304
# gate/up tiles leave 48 (halves in 2 pieces), 152 down-dgrad tiles (no cut);
# 158 gate/up tiles (no cut), 79 down-dgrad tiles (halves); 102 tiles of
# either, the down dgrad's 128 wide (halves; 2 pieces); 64 and 32 tiles
# (halves; halves in 3 pieces); 40 and 20 tiles (halves in 2 and in 4
# pieces); 66 and 42 tiles, the down dgrad's 128 wide (3 and 4 pieces)
@pytest.mark.parametrize("F,rows,layout", [
    (256, [9000, 20000, 9400], ((2, 2), (1, 1))),
    (256, [5000, 12000, 3000], ((1, 1), (2, 1))),
    (384, [2000, 5000, 1500], ((2, 1), (1, 2))),
    (256, [4000, 4000], ((2, 1), (2, 3))),
    (256, [3000, 2000], ((2, 2), (2, 4))),
    (384, [3000, 2500], ((2, 1), (1, 3))),
    (384, [2000, 1500], ((2, 2), (1, 4))),
], ids=["rounds+tail", "halves", "128-wide-tiles", "halves-3-pieces", "halves-4-pieces", "128-wide-3-pieces",
        "128-wide-4-pieces"])
def test_tail_split_parity_and_determinism(gpu, F, rows, layout):
    from paper_2606_11867_amd import api
    grid = torch.cuda.get_device_properties(gpu).multi_processor_count
    l_fwd = expected_layout(rows, 2 * F, D, grid)   # gate/up forward: N = 2F, K = d
    l_dgr = expected_layout(rows, F, D, grid)       # down dgrad: N = F, K = d
    print(f"F={F} rows {rows}: (halves, pieces) gate/up fwd {l_fwd}, down dgrad {l_dgr} ({grid} CUs)", flush=True)
    assert (l_fwd, l_dgr) != ((1, 1), (1, 1)), "layout no longer exercises the cuts"
    if grid == 256:
        assert (l_fwd, l_dgr) == layout
    rng = np.random.default_rng(5)
    off = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    N = int(off[-1])
    x = bf16_round(rng.standard_normal((N, D)).astype(np.float32))
    dy = bf16_round(rng.standard_normal((N, D)).astype(np.float32))
    gu = bf16_round((rng.standard_normal((W, 2 * F, D)) / np.sqrt(D)).astype(np.float32))
    dn = bf16_round((rng.standard_normal((W, D, F)) / np.sqrt(F)).astype(np.float32))
    # saved [A | U] for the input gradient: seeded inputs of their own (the
    # forward's are checked against the oracle separately)
    au_in = bf16_round((2.0 * rng.standard_normal((N, 2 * F))).astype(np.float32))
    widx = (np.arange(len(rows)) % W).astype(np.int32)
    bf = torch.bfloat16
    dev = lambda a: torch.from_numpy(a).to(gpu).to(bf)  # noqa: E731
    xd, dyd, gud, dnd, aud = dev(x), dev(dy), dev(gu), dev(dn), dev(au_in)
    so = torch.from_numpy(off).to(gpu)
    wi = torch.from_numpy(widx).to(gpu)
    ws = api.ffn_workspace(gpu)

    runs = []
    for w_ in (ws, ws, None):
        h, y, au = api.grouped_ffn_fwd(xd, so, wi, gud, dnd, ws=w_)
        d_au, dx = api.grouped_ffn_dgrad(dyd, aud, so, wi, gud, dnd, ws=w_)
        runs.append(dict(h=h, y=y, au=au, d_au=d_au, dx=dx))
    torch.cuda.synchronize()
    assert not ws[:4096].any().item(), "split arrival counters not reset"
    for k in runs[0]:
        assert torch.equal(runs[0][k], runs[1][k]), f"{k}: split result not deterministic"
        check_close(f"{k} split vs unsplit", to_np(runs[0][k]), to_np(runs[2][k]))

    # sampled rows of every slot against the oracle
    r, sub, sw = sampled(off, rng)
    f = O.ffn_forward(x[r].astype(np.float64), sub, sw, gu, dn)
    rt = torch.from_numpy(r).to(gpu)
    check_close("H", to_np(runs[0]["h"][rt]), f["H"])
    check_close("Y", to_np(runs[0]["y"][rt]), f["Y"])
    check_close("A", to_np(runs[0]["au"][rt][:, :F]), f["A"])
    check_close("U", to_np(runs[0]["au"][rt][:, F:]), f["U"])
    g = O.ffn_dgrad(dy[r].astype(np.float64), au_in[r, :F], au_in[r, F:], sub, sw, gu, dn)
    check_close("dA", to_np(runs[0]["d_au"][rt][:, :F]), g["dA"])
    check_close("dU", to_np(runs[0]["d_au"][rt][:, F:]), g["dU"])
    check_close("dX", to_np(runs[0]["dx"][rt]), g["dX"])


# (F, rows): d = 2048, so both plain-store GEMMs (down forward, K = F, and
# gate/up dgrad, K = 2F) have 8 columns of tiles. 66 m-tiles (528 tiles: two
# whole rounds and 16 tiles cut into 32 halves); 11 m-tiles (88 tiles, all
# halves); F = 2048 and 7 m-tiles (56 tiles of 32 and 64 k-steps: halves
# without a workspace, halves in 2 K pieces with one)
@pytest.mark.parametrize("F,rows", [(768, [9000, 7000, 300]), (768, [2000, 700]), (2048, [1000, 700])],
                         ids=["rounds+halves", "all-halves", "long-k"])
def test_n_split_last_round(gpu, F, rows):
    from paper_2606_11867_amd import api
    grid = torch.cuda.get_device_properties(gpu).multi_processor_count
    cases = {(g, ws): expected_layout(rows, D, k, grid, ws)
             for g, k in (("down_fwd", F), ("gate_up_dgrad", 2 * F)) for ws in (False, True)}
    print(f"F={F} rows {rows}: (halves, pieces) {cases} ({grid} CUs)", flush=True)
    if grid == 256:
        assert all(v[0] == 2 for v in cases.values()), "layout no longer cuts along N"
        assert (cases[("down_fwd", True)][1] == 2) == (F == 2048)
    rng = np.random.default_rng(17)
    off = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    N = int(off[-1])
    x = bf16_round(rng.standard_normal((N, D)).astype(np.float32))
    dy = bf16_round(rng.standard_normal((N, D)).astype(np.float32))
    gu = bf16_round((rng.standard_normal((W, 2 * F, D)) / np.sqrt(D)).astype(np.float32))
    dn = bf16_round((rng.standard_normal((W, D, F)) / np.sqrt(F)).astype(np.float32))
    au_in = bf16_round((2.0 * rng.standard_normal((N, 2 * F))).astype(np.float32))
    widx = (np.arange(len(rows)) % W).astype(np.int32)
    bf = torch.bfloat16
    dev = lambda a: torch.from_numpy(a).to(gpu).to(bf)  # noqa: E731
    xd, dyd, gud, dnd, aud = dev(x), dev(dy), dev(gu), dev(dn), dev(au_in)
    so = torch.from_numpy(off).to(gpu)
    wi = torch.from_numpy(widx).to(gpu)
    ws = api.ffn_workspace(gpu)
    runs = []
    for w_ in (None, None, ws):
        h, y, au = api.grouped_ffn_fwd(xd, so, wi, gud, dnd, ws=w_)
        d_au, dx = api.grouped_ffn_dgrad(dyd, aud, so, wi, gud, dnd, ws=w_)
        runs.append(dict(h=h, y=y, au=au, d_au=d_au, dx=dx))
    torch.cuda.synchronize()
    assert not ws[:4096].any().item(), "split arrival counters not reset"
    for k in runs[0]:
        assert torch.equal(runs[0][k], runs[1][k]), f"{k}: not deterministic"
        check_close(f"{k} without vs with workspace", to_np(runs[0][k]), to_np(runs[2][k]))
    # the down forward and the gate/up dgrad against the oracle: every row
    # when the oracle is quick, else sampled rows of every slot
    if N <= 4000:
        r, sub, sw = np.arange(N), off, widx
    else:
        r, sub, sw = sampled(off, rng)
    f = O.ffn_forward(x[r].astype(np.float64), sub, sw, gu, dn)
    g = O.ffn_dgrad(dy[r].astype(np.float64), au_in[r, :F], au_in[r, F:], sub, sw, gu, dn)
    rt = torch.from_numpy(r).to(gpu)
    for i, run in enumerate((runs[0], runs[2])):
        check_close(f"Y (run {i})", to_np(run["y"][rt]), f["Y"])
        check_close(f"dX (run {i})", to_np(run["dx"][rt]), g["dX"])
        check_close(f"H (run {i})", to_np(run["h"][rt]), f["H"])
        check_close(f"dA (run {i})", to_np(run["d_au"][rt][:, :F]), g["dA"])


def test_invalid_weight_index_slot_is_skipped(gpu):
    """A slot whose weight index is outside [0, W) is skipped by every row
    GEMM: its rows of every output keep what they held, and no arrival
    counter is left set, also when the last round is cut into halves and K
    pieces (here halves in 2 pieces for the gate/up forward, in 4 for the
    down dgrad); the other slots' rows match the oracle."""
    from paper_2606_11867_amd import _lib, api
    F, rows, widx = 256, [3000, 2000, 700], [0, -1, W]
    grid = torch.cuda.get_device_properties(gpu).multi_processor_count
    if grid == 256:
        assert expected_layout(rows, 2 * F, D, grid) == (2, 2) and expected_layout(rows, F, D, grid) == (2, 4)
    rng = np.random.default_rng(23)
    off = np.concatenate([[0], np.cumsum(rows)]).astype(np.int32)
    N = int(off[-1])
    x = bf16_round(rng.standard_normal((N, D)).astype(np.float32))
    dy = bf16_round(rng.standard_normal((N, D)).astype(np.float32))
    gu = bf16_round((rng.standard_normal((W, 2 * F, D)) / np.sqrt(D)).astype(np.float32))
    dn = bf16_round((rng.standard_normal((W, D, F)) / np.sqrt(F)).astype(np.float32))
    au_in = bf16_round((2.0 * rng.standard_normal((N, 2 * F))).astype(np.float32))
    bf = torch.bfloat16
    dev = lambda a: torch.from_numpy(a).to(gpu).to(bf)  # noqa: E731
    xd, dyd, gud, dnd, aud = dev(x), dev(dy), dev(gu), dev(dn), dev(au_in)
    so = torch.from_numpy(off).to(gpu)
    wi = torch.from_numpy(np.array(widx, dtype=np.int32)).to(gpu)
    ws = api.ffn_workspace(gpu)
    sentinel = 7.0
    h, y, au = (torch.full((N, c), sentinel, dtype=bf, device=gpu) for c in (F, D, 2 * F))
    d_au, dx = (torch.full((N, c), sentinel, dtype=bf, device=gpu) for c in (2 * F, D))
    lib = _lib.load()
    st = torch.cuda.current_stream(gpu).cuda_stream
    print(f"\n[case] slots {rows} with weight indices {widx} (W={W}), F={F}", flush=True)
    assert lib.foremoe_grouped_ffn_fwd(xd.data_ptr(), _lib.BF16, D, F, len(rows), so.data_ptr(), wi.data_ptr(), W,
                                       gud.data_ptr(), dnd.data_ptr(), N, h.data_ptr(), y.data_ptr(), au.data_ptr(),
                                       ws.data_ptr(), ws.numel(), st) == 0
    assert lib.foremoe_grouped_ffn_dgrad(dyd.data_ptr(), aud.data_ptr(), _lib.BF16, D, F, len(rows), so.data_ptr(),
                                         wi.data_ptr(), W, gud.data_ptr(), dnd.data_ptr(), N, d_au.data_ptr(),
                                         dx.data_ptr(), ws.data_ptr(), ws.numel(), st) == 0
    torch.cuda.synchronize()
    assert not ws[:4096].any().item(), "split arrival counters not reset"
    skipped = slice(int(off[1]), N)  # slots 1 and 2
    for name, t in (("H", h), ("Y", y), ("A|U", au), ("dA|dU", d_au), ("dX", dx)):
        assert bool((t[skipped] == sentinel).all()), f"{name}: rows of a skipped slot were written"
    n0 = int(off[1])
    sub, sw = np.array([0, n0]), np.array([0])
    f = O.ffn_forward(x[:n0].astype(np.float64), sub, sw, gu, dn)
    g = O.ffn_dgrad(dy[:n0].astype(np.float64), au_in[:n0, :F], au_in[:n0, F:], sub, sw, gu, dn)
    check_close("H (slot 0)", to_np(h[:n0]), f["H"])
    check_close("Y (slot 0)", to_np(y[:n0]), f["Y"])
    check_close("dA (slot 0)", to_np(d_au[:n0, :F]), g["dA"])
    check_close("dX (slot 0)", to_np(dx[:n0]), g["dX"])
