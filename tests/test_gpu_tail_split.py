"""Row GEMMs with the optional workspace: a partial last round of output
tiles is cut along K into up to 4 pieces whose fp32 partial sums the last
piece to finish adds in piece order (grouped SwiGLU FFN of App. A; the
split only changes the fp32 summation order of the Step-4 products).

Row layouts are chosen so that the split really happens (the expected
piece count per GEMM is computed here from the tile counts and asserted
non-trivial): one with whole rounds of tiles plus a split tail, one with
fewer tiles than workgroups (every tile split), one where the down dgrad
runs on 128-wide output tiles (F not a multiple of 256). Checked: sampled rows
against the fp64 oracle, split against unsplit within the tolerance, two
split runs bit for bit equal, and the arrival counters left at zero.
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


def expected_split(rows, n_cols, k, grid):
    """Pieces per tile of the last round (1: no split), as the kernel picks them
    (256-wide output tiles when n_cols allows, else 128-wide): as many as keep
    at most 7/8 of the workgroups busy, at most SPLIT_MAX."""
    bn = 256 if n_cols % 256 == 0 else 128
    tiles = sum((r + 255) // 256 for r in rows) * (n_cols // bn)
    rem = tiles % grid
    if rem == 0 or k // 64 < SPLIT_MIN_K:
        return 1
    s = min((7 * grid // 8) // rem, SPLIT_MAX)
    return s if s >= 2 else 1


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


# (F, rows of each slot, expected pieces of the gate/up forward and the down
# dgrad on a 256-CU MI355X): 304 gate/up tiles leave a last round of 48 (4
# pieces); 79 down-dgrad tiles (2 pieces); 102 tiles of either (2 pieces);
# 64 gate/up tiles (3 pieces) and 32 down-dgrad tiles (4 pieces)
@pytest.mark.parametrize("F,rows,pieces", [(256, [9000, 20000, 9400], (4, 1)), (256, [5000, 12000, 3000], (1, 2)),
                                           (384, [2000, 5000, 1500], (2, 2)), (256, [4000, 4000], (3, 4))],
                         ids=["rounds+tail", "all-split", "128-wide-tiles", "three-and-four-pieces"])
def test_tail_split_parity_and_determinism(gpu, F, rows, pieces):
    from paper_2606_11867_amd import api
    grid = torch.cuda.get_device_properties(gpu).multi_processor_count
    s_fwd = expected_split(rows, 2 * F, D, grid)   # gate/up forward: N = 2F, K = d
    s_dgr = expected_split(rows, F, D, grid)       # down dgrad: N = F, K = d
    print(f"F={F} rows {rows}: pieces gate/up fwd {s_fwd}, down dgrad {s_dgr} ({grid} CUs)", flush=True)
    assert max(s_fwd, s_dgr) >= 2, "layout no longer exercises the split"
    if grid == 256:
        assert (s_fwd, s_dgr) == pieces
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
