"""The single-pass schedule (lamb_tile_schedule, host only): every layer's
tiles cover it exactly, sit consecutively inside one round, and a simulation
of the persistent grid's waits always runs to the end."""

import numpy as np
import pytest

from paper_1904_00962_amd import _lib, paramsets

TILE = 8192


def _check_layout(numel, round_):
    et, es, el, first, tiles = _lib.lamb_tile_schedule(numel, round_)
    n = len(et)
    seen = [False] * n
    for i, size in enumerate(numel):
        nt = -(-size // TILE)
        if nt > round_:
            assert tiles[i] == 0, "layer %d of %d tiles must take the two-pass path" % (i, nt)
            continue
        assert tiles[i] == nt
        f = first[i]
        assert f // round_ == (f + nt - 1) // round_, "layer %d straddles a round" % i
        for k in range(nt):
            j = f + k
            assert not seen[j]
            seen[j] = True
            assert et[j] == i and es[j] == k * TILE and el[j] == min(TILE, size - k * TILE)
    for j in range(n):
        if not seen[j]:  # an empty entry: only in a gap at the end of a full round
            assert et[j] == -1 and el[j] == 0
            assert j // round_ < (n - 1) // round_
            assert all(not seen[k] for k in range(j, (j // round_ + 1) * round_))
    return et, first, tiles


def _simulate(et, first, tiles, round_):
    """The kernel's schedule step by step: workgroup w takes entries w, w + G,
    ... in order; a tile publishes its partial without waiting; the layer's
    leader waits for every partial, a member for the leader's scale."""
    n = len(et)
    G = min(n, round_)
    pos = list(range(G))
    published = [False] * n
    scale = {}
    steps = 0
    while any(p < n for p in pos):
        progress = False
        for w in range(G):
            j = pos[w]
            if j >= n:
                continue
            i = et[j]
            if i < 0:
                pos[w] += G
                progress = True
                continue
            if not published[j]:
                published[j] = True
                progress = True
            f, t = first[i], tiles[i]
            if j == f:
                if all(published[f:f + t]):
                    scale[i] = True
                    pos[w] += G
                    progress = True
            elif scale.get(i):
                pos[w] += G
                progress = True
        steps += 1
        assert progress, "the grid would wait forever (entries %s)" % sorted(set(pos))
    return steps


@pytest.mark.parametrize("cfg", range(5))
def test_paramset_schedules(cfg):
    ps = paramsets.get(cfg)
    numel = [t.numel for t in ps.tensors]
    et, first, tiles = _check_layout(numel, 1024)
    _simulate(et, first, tiles, 1024)


def test_bert_large_packs_without_padding():
    """BERT-Large on 256 CUs: every layer but the token embedding takes the
    single pass, in 37 rounds with no empty entry."""
    ps = paramsets.get(2)
    numel = [t.numel for t in ps.tensors]
    et, first, tiles = _check_layout(numel, 1024)
    assert sum(1 for k in tiles if k == 0) == 1
    assert -1 not in et
    assert -(-len(et) // 1024) == 37


@pytest.mark.parametrize("seed", range(12))
def test_random_layers_small_rounds(seed):
    rng = np.random.default_rng(seed)
    round_ = int(rng.integers(1, 40))
    n = int(rng.integers(1, 60))
    numel = [int(v) for v in rng.integers(1, TILE * (round_ + 3), size=n)]
    numel += [TILE * round_, TILE * round_ + 1, 1, TILE]
    et, first, tiles = _check_layout(numel, round_)
    if et:
        _simulate(et, first, tiles, round_)


def test_round_boundary_and_errors():
    et, es, el, first, tiles = _lib.lamb_tile_schedule([TILE * 4, TILE * 4 + 1, 5], 4)
    assert tiles == [4, 0, 1] and first == [0, 0, 4] and len(et) == 5
    with pytest.raises(_lib.LambError):
        _lib.lamb_tile_schedule([TILE], 0)
    with pytest.raises(_lib.LambError):
        _lib.lamb_tile_schedule([0], 4)
