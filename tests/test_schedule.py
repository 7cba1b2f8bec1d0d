"""The single-pass schedule (lamb_tile_schedule, host only): every layer's
tiles cover it exactly, sit consecutively inside one round, and a simulation
of the persistent grid's waits always runs to the end. A plan's tile shape is
the wide one (10 groups of 1024 elements) exactly when that puts more
parameters on the single pass than the narrow one (8 groups)."""

import numpy as np
import pytest

from paper_1904_00962_amd import _lib, paramsets

TILE = 8192
BLOCK = 1024
NARROW, WIDE = 8, 10


def _single_pass_params(numel, max_round, groups):
    return sum(n for n in numel if -(-n // (groups * BLOCK)) <= max_round)


def _check_layout(numel, max_round, tile_groups=0):
    et, es, el, first, tiles, round_, groups = _lib.lamb_tile_schedule(numel, max_round,
                                                                      tile_groups)
    if tile_groups:
        assert groups == tile_groups
    else:
        wide = _single_pass_params(numel, max_round, WIDE)
        assert groups == (WIDE if wide > _single_pass_params(numel, max_round, NARROW) else NARROW)
    tile = groups * BLOCK
    n = len(et)
    assert 1 <= round_ <= max_round
    n_rounds = -(-n // round_)
    # the last round holds at least one entry; the rounds hold every tile
    real = sum(tiles)
    assert n == 0 or n > (n_rounds - 1) * round_
    assert real <= n and n_rounds >= -(-real // max_round)
    assert all(k <= round_ for k in tiles)
    seen = [False] * n
    for i, size in enumerate(numel):
        nt = -(-size // tile)
        if nt > max_round:
            assert tiles[i] == 0, "layer %d of %d tiles must take the two-pass path" % (i, nt)
            continue
        assert tiles[i] == nt
        f = first[i]
        assert f // round_ == (f + nt - 1) // round_, "layer %d straddles a round" % i
        covered = 0
        for k in range(nt):
            j = f + k
            assert not seen[j]
            seen[j] = True
            # tile k holds the 1024-element blocks k, k + nt, ..., k + (groups - 1) nt
            held = sum(max(0, min(BLOCK, size - b * BLOCK)) for b in range(k, groups * nt, nt))
            assert et[j] == i and es[j] == k * BLOCK and el[j] == held > 0
            covered += held
        assert covered == size
    for j in range(n):
        if not seen[j]:  # an empty entry: only in a gap at the end of a full round
            assert et[j] == -1 and el[j] == 0
            assert j // round_ < (n - 1) // round_
            assert all(not seen[k] for k in range(j, (j // round_ + 1) * round_))
    return et, first, tiles, round_, groups


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
    et, first, tiles, round_, _ = _check_layout(numel, 1024)
    _simulate(et, first, tiles, round_)


def test_bert_large_layout():
    """BERT-Large on 256 CUs: every layer but the token embedding takes the
    single pass, in 37 rounds with no empty entry. Two 512-tile FFN layers
    fill a round, so no narrower round would do."""
    ps = paramsets.get(2)
    numel = [t.numel for t in ps.tensors]
    et, first, tiles, round_, groups = _check_layout(numel, 1024)
    assert groups == NARROW and sum(1 for k in tiles if k == 0) == 1
    assert round_ == 1024 and -(-len(et) // round_) == 37 and -1 not in et


def test_resnet50_rounds_are_balanced():
    """ResNet-50's 3223 tiles need four rounds; they are packed four about
    equal rounds instead of three full ones and a short one."""
    ps = paramsets.get(3)
    numel = [t.numel for t in ps.tensors]
    et, first, tiles, round_, groups = _check_layout(numel, 1024)
    assert groups == NARROW and -(-len(et) // round_) == 4 and sum(tiles) == 3223
    assert round_ < 900


def test_gpt_1p5b_takes_wide_tiles():
    """The 1.5B set's 10.24M-element FFN layers need 1250 narrow tiles but
    only 1000 wide ones: with wide tiles they join the single pass, and only
    the token embedding stays on the two-pass kernels."""
    ps = paramsets.get(4)
    numel = [t.numel for t in ps.tensors]
    et, first, tiles, round_, groups = _check_layout(numel, 1024)
    assert groups == WIDE
    two_pass = [n for n, k in zip(numel, tiles) if k == 0]
    assert two_pass == [max(numel)] and max(numel) > WIDE * BLOCK * 1024
    ffn = [k for n, k in zip(numel, tiles) if n == 1600 * 6400]
    assert ffn and all(k == 1000 for k in ffn)
    _, _, narrow_tiles, _, _ = _check_layout(numel, 1024, NARROW)
    assert all(k == 0 for n, k in zip(numel, narrow_tiles) if n == 1600 * 6400)


@pytest.mark.parametrize("tile_groups", [0, NARROW, WIDE])
@pytest.mark.parametrize("seed", range(12))
def test_random_layers_small_rounds(seed, tile_groups):
    rng = np.random.default_rng(seed)
    round_ = int(rng.integers(1, 40))
    n = int(rng.integers(1, 60))
    numel = [int(v) for v in rng.integers(1, TILE * (round_ + 3), size=n)]
    numel += [TILE * round_, TILE * round_ + 1, 1, TILE, WIDE * BLOCK * round_ + 1]
    et, first, tiles, width, _ = _check_layout(numel, round_, tile_groups)
    if et:
        _simulate(et, first, tiles, width)


def test_round_boundary_and_errors():
    sizes = [TILE * 4, TILE * 4 + 1, 5]
    et, es, el, first, tiles, width, groups = _lib.lamb_tile_schedule(sizes, 4, NARROW)
    assert tiles == [4, 0, 1] and first == [0, 0, 4] and len(et) == 5 and width == 4
    # the wide tile takes the second layer too (4 tiles of 10240), so a plan
    # picks it: rounds {4}, {4}, {1}
    et, es, el, first, tiles, width, groups = _lib.lamb_tile_schedule(sizes, 4)
    assert groups == WIDE and tiles == [4, 4, 1] and width == 4 and len(et) == 9
    # three layers of 3, 3 and 2 tiles fill two rounds of 6 as {3, 3}, {2}; the
    # narrowest width that still needs two rounds is 5: {3, 2}, {3}
    et, es, el, first, tiles, width, groups = _lib.lamb_tile_schedule(
        [3 * TILE, 3 * TILE, 2 * TILE], 6)
    assert groups == NARROW and width == 5 and tiles == [3, 3, 2] and len(et) == 8
    assert et == [0, 0, 0, 2, 2, 1, 1, 1]
    with pytest.raises(_lib.LambError):
        _lib.lamb_tile_schedule([TILE], 0)
    with pytest.raises(_lib.LambError):
        _lib.lamb_tile_schedule([0], 4)
    with pytest.raises(_lib.LambError):
        _lib.lamb_tile_schedule([TILE], 4, 9)
