"""CPU replay of the persistent launch (the fused kernel's PERSIST variant).

The kernel's rules are restated here from its definition, independently of
the library, and replayed for plans that the library runs persistent:

* Assignment.  The plain launch order (no split key ranges) has one
  workgroup per query tile; its workgroups b = 8 i + x (XCD x) become the
  items of XCD x, shared by the launch's S = grid / 8 workgroups on that XCD
  in rounds: in round r slot s takes item r S + s when r is even and
  r S + S - 1 - s when r is odd.  Every query tile must be taken exactly once.
* Waits.  One ring of K/V tiles runs through all of a workgroup's query
  tiles.  Per wave, in issue order: the copies of tile 0, the first query
  tile's Q loads, the copies of tiles 1 and 2; then in step j the next query
  tile's Q loads (when a switch comes at step j + 2), the copies of tile
  j + 3, the finished query tile's stores (at a switch), and a wait for the
  copies of tile j + 1.  Vector memory operations complete in issue order,
  so the wait must allow at most the operations issued after tile j + 1's
  last copy.  The kernel allows 4 LPW (two tiles of copies), plus QL in the
  two steps before a switch and NST in the switch step and the two after it.
  The replay counts the exact number at every step of every workgroup: the
  rule never allows more (it would stop waiting too early), and it allows
  fewer only where two switches are 4 steps apart.
"""
import pytest

from paper_2609_10937_amd import capi

WAVES = 8
AHEAD = 2  # tiles requested ahead of the one being computed (5 LDS stages)


def _order(BH, n_qt):
    """The fused kernel's workgroup order without split key ranges."""
    xg = 1
    while xg * n_qt < 64:
        xg *= 2
    return ("units" if BH % (8 * xg) == 0 else "plain"), xg


def _decode(b, BH, n_qt, causal, order, xg):
    """Workgroup b of the plain launch order -> (head, query tile)."""
    if order == "units":
        x, i = b % 8, b // 8
        per_group = xg * n_qt
        gi, r = divmod(i, per_group)
        rank = r // xg
        head = x + 8 * (gi * xg + (r - rank * xg))
    else:
        rank, head = divmod(b, BH)
    return head, (n_qt - 1 - rank if causal else rank)


def _tiles(qt, L, tile_q, t_kv, causal):
    n = -(-L // t_kv)
    return min(n, -(-min(L, (qt + 1) * tile_q) // t_kv)) if causal else n


def _assignment(BH, L, tile_q, t_kv, causal, grid):
    n_qt = -(-L // tile_q)
    order, xg = _order(BH, n_qt)
    S = grid // 8
    taken = {}
    per_wg = []
    for blk in range(grid):
        x, s = blk % 8, blk // 8
        items = (BH * n_qt - x + 7) // 8
        units = []
        r = 0
        while True:
            it = r * S + (S - 1 - s if r % 2 else s)
            if it >= items:
                break
            b = 8 * it + x
            head, qt = _decode(b, BH, n_qt, causal, order, xg)
            assert 0 <= head < BH and 0 <= qt < n_qt
            assert (head, qt) not in taken, f"query tile {(head, qt)} taken twice"
            taken[(head, qt)] = blk
            units.append(_tiles(qt, L, tile_q, t_kv, causal))
            r += 1
        per_wg.append(units)
    assert len(taken) == BH * n_qt
    return per_wg, order


def _replay_waits(units, lpw, ql, nst, allow=None):
    """Replay one workgroup's vector memory operations (ql Q loads per query
    tile, nst stores per finished query tile); return the number of waits
    checked and the (step, tiles of the current and the previous query tile)
    of every wait that allows fewer operations than it could.  `allow` =
    (Q-load term, store term) of the wait rule, the kernel's by default."""
    ql_a, nst_a = allow if allow is not None else (ql, nst)
    n_ops = 0
    last_copy = {}

    def copies(t):
        nonlocal n_ops
        n_ops += 2 * lpw
        last_copy[t] = n_ops - 1

    copies(0)
    n_ops += ql  # the first query tile's Q rows
    for t in range(1, AHEAD + 1):
        copies(t)
    cur, nx_start = 0, units[0]
    last_switch = -8
    checks, conservative = 0, []

    def wait(j):
        nonlocal checks
        nx_valid = cur + 1 < len(units)
        e = j - (nx_start if nx_valid and nx_start - j <= 2 else last_switch)
        allowed = 4 * lpw + (ql_a if -2 <= e < 0 else 0) + (nst_a if 0 <= e <= 2 else 0)
        exact = n_ops - 1 - last_copy[j + 1]
        assert allowed <= exact, f"step {j}: the wait allows {allowed} operations, {exact} follow the tile"
        if allowed < exact:
            conservative.append((j, units[cur], units[cur - 1] if cur else None))
        checks += 1

    copies(AHEAD + 1)
    wait(0)
    j = 1
    while True:
        nx_valid = cur + 1 < len(units)
        if j == nx_start and not nx_valid:
            break
        if nx_valid and j + 2 == nx_start:
            n_ops += ql
        copies(j + AHEAD + 1)
        if j == nx_start:
            n_ops += nst
            cur += 1
            nx_start = j + units[cur]
            last_switch = j
        wait(j)
        j += 1
    assert j == sum(units)
    return checks, conservative


SHAPES = [
    # B, H, L, d, causal
    (1, 1024, 512, 128, False),
    (1, 1024, 200, 128, False),
    (1, 300, 700, 128, False),
    (1, 512, 1024, 128, True),
    (1, 520, 256, 128, True),
    (4, 64, 512, 128, False),
    (1, 1024, 512, 64, False),
    (2, 160, 512, 64, False),
    (1, 288, 1024, 128, True),
    (3, 101, 777, 128, True),
]


@pytest.mark.parametrize("B,H,L,d,causal", SHAPES)
def test_persistent_schedule_replay(B, H, L, d, causal):
    hw = capi.attn_hw_desc_preset("gfx950")
    r = capi.attn_fwd_plan(B, H, L, d, causal, capi.ATTN_BF16, hw=hw)
    assert r.launch_grid < r.grid, "shape expected to run persistent"
    assert r.n_waves == WAVES and r.n_split == 1
    per_wg, _ = _assignment(B * H, L, r.tile_q, r.t_kv, causal, r.launch_grid)
    qb = r.t_q_wave // 16
    lpw = r.t_kv * d * 2 // 1024 // WAVES  # 1 KB copy blocks per wave per K (or V) tile
    ql, nst = qb * d // 32, qb * d // 16    # 16-byte Q loads and 8-byte stores per lane
    total = 0
    for units in per_wg:
        if not units:
            continue
        assert min(units) >= AHEAD + 2
        checks, conservative = _replay_waits(units, lpw, ql, nst)
        total += checks
        # conservative only where a query tile of 4 key tiles puts two switches
        # 4 steps apart (the stores after one overlap the Q loads before the next)
        for j, here, before in conservative:
            assert here == 4 and before is not None, (j, here, before)
    assert total == sum(sum(u) for u in per_wg)
    # no workgroup carries more than one query tile's work above the mean
    loads = [sum(u) for u in per_wg]
    longest = max(max(u) for u in per_wg if u)
    assert max(loads) <= sum(loads) / len(loads) + longest


def test_replay_catches_a_short_wait():
    """A rule that counted one store or Q load more than are issued would let
    the wave go on before the awaited tile's copies have landed: the replay
    must notice, while the kernel's own counts pass."""
    _replay_waits([4, 5, 4], lpw=2, ql=8, nst=16)
    with pytest.raises(AssertionError):
        _replay_waits([4, 5, 4], lpw=2, ql=8, nst=16, allow=(8, 17))
    with pytest.raises(AssertionError):
        _replay_waits([5, 6, 4], lpw=2, ql=8, nst=16, allow=(9, 16))
