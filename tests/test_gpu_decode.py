"""Decode-batch shapes, held bit for bit to the training-mode ones.

Decode batches (rollout mode) take half vocabulary tiles -- one vocab wave
per workgroup, a partial per 128-entry half of each tile, the two halves
merged (lower first) in the merge pass -- always for 65..128 rows (two
workgroups per CU against one), and up to 64 rows where they fill the chip's
rounds more evenly than whole tiles (V = 151936 on 256 CUs: 1187 halves on
768 slots against 594 tiles on 512). Launches of at most 512 rows merge with
four waves per row. The tests cover vocabulary sizes whose last tile is
whole, has a partial upper half, only a lower half, or a partial lower half,
tokens in every lane-group position of both halves and in the last tile, and
the fp64 oracle."""

import numpy as np
import pytest
import torch

import paper_2605_14220_amd as tim
from paper_2605_14220_amd import Mode
from tim_testutil import TOL_ENT, TOL_LOGP, bits_equal, check_close, inputs, oracle_rows, random_tokens, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _tokens(T, V, seed):
    """Random tokens, with the first rows on the edges of halves and tiles:
    entries 16 b + 4 g + r of either half for several lane groups g, the first
    and last entry of each half, and the last entries of V."""
    tok = random_tokens(T, V, seed).cpu()
    edge = [0, 3, 4, 15, 16, 127, 128, 131, 132, 143, 255, 256, 383, 384, 511, V - 129, V - 128, V - 2, V - 1]
    edge = [v for v in edge if 0 <= v < V]
    n = min(T, len(edge))
    tok[:n] = torch.tensor(edge[:n], dtype=torch.int32)
    return tok.cuda()


def _same(a, b):
    for x, y in zip(a, b):
        assert bits_equal(x, y)


def _fill(units, slots):
    return units / (-(-units // slots) * slots)


def _per_row(V, T):
    """Partials per row of the planner's choice on this device: halves above
    64 rows; up to 64, half tiles (3 workgroups per CU) when their last round
    leaves fewer slots idle than whole tiles (2 per CU), else whole tiles."""
    nv, nh = -(-V // 256), -(-V // 128)
    if T > 64:
        return nh
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    return nh if _fill(nh, 3 * cus) > _fill(nv, 2 * cus) else nv


def _shape(V, T):
    return "half" if _per_row(V, T) == -(-V // 128) else "whole"


def _decode(h, W, tok, tau):
    """Rollout call through a workspace pre-filled with 0xFF: returns the
    outputs and the number of 16-byte partials the call wrote per row, which
    names the shape that ran (ceil(V / 128) for half tiles, ceil(V / 256) for
    whole ones)."""
    T, d = h.shape
    V = W.shape[0]
    ws = torch.full((tim.workspace_size(T, d, V, Mode.ROLLOUT),), 255, dtype=torch.uint8, device="cuda")
    out = tim.logprobs(h, W, tok, tau, mode=Mode.ROLLOUT, lse=True, workspace=ws)
    rec = ws.view(-1, 16)
    written = int((rec != 255).any(dim=1).sum().item())
    assert written % T == 0
    return out, written // T


@pytest.mark.parametrize("V", [1, 2, 127, 128, 129, 255, 256, 257, 383, 384, 385, 4096 + 77, 4096 + 200,
                               151936, 152064, 512 * 256 + 77, 512 * 256 + 200, 600 * 256])
@pytest.mark.parametrize("T", [1, 19, 64, 65, 100, 128])
def test_decode_bitwise_equal_whole_tiles(V, T):
    d = 256
    print(f"case halves V={V} T={T}", flush=True)
    h, W = inputs(T, d, V, seed=V % 1000 + T, w_std=0.1)
    tok = _tokens(T, V, seed=V + T)
    dec, per_row = _decode(h, W, tok, 0.7)
    assert per_row == _per_row(V, T)
    print(f"  {_shape(V, T)} tiles, {per_row} partials per row", flush=True)
    trn = tim.logprobs(h, W, tok, 0.7, mode=Mode.TRAINING, lse=True)        # whole tiles
    _same(dec, trn)
    if V <= 4096 + 200:
        ref_lp, ref_H = oracle_rows(h, W, tok, 0.7)
        check_close(f"halves logp V={V}", dec[0], ref_lp, TOL_LOGP)
        check_close(f"halves entropy V={V}", dec[1], ref_H, TOL_ENT)


def test_halves_full_size_rows_against_oracle():
    """d = 4096, V = 151936, a decode batch of 64 rows: bitwise equal to the
    training path and within tolerance of the oracle on every row."""
    T, d, V = 64, 4096, 151936
    h, W = inputs(T, d, V, seed=41, w_std=0.02)
    tok = _tokens(T, V, seed=41)
    dec, per_row = _decode(h, W, tok, 1.0)
    if torch.cuda.get_device_properties(0).multi_processor_count == 256:
        assert per_row == 1187      # 1187 halves on 768 slots beat 594 tiles on 512
    else:
        assert per_row == _per_row(V, T)
    trn = tim.logprobs(h, W, tok, 1.0, mode=Mode.TRAINING, lse=True)
    _same(dec, trn)
    ref_lp, ref_H = oracle_rows(h, W, tok, 1.0)
    check_close("decode logp", dec[0], ref_lp, TOL_LOGP)
    check_close("decode entropy", dec[1], ref_H, TOL_ENT)


def test_halves_gather_is_bit_exact():
    """logp = z_tok - lse bit for bit, z from the logits dump (whole tiles),
    with the token at each of the 128 entries of both halves of a tile."""
    T, d, V = 64, 256, 1000
    h, W = inputs(T, d, V, seed=42)
    for base in (256, 384):
        tok = (torch.arange(T, dtype=torch.int32) * 2 + base + (1 if base == 384 else 0)).cuda()
        (lp, _, lse), per_row = _decode(h, W, tok, 0.8)
        assert per_row == _per_row(V, T)
        z = tim.logits(h, W, 0.8)
        ztok = z.gather(1, tok.long()[:, None])[:, 0]
        assert bits_equal(lp, ztok - lse)


def test_halves_out_of_range_tokens():
    T, d, V = 20, 256, 1000
    h, W = inputs(T, d, V, seed=43)
    tok = random_tokens(T, V, seed=43)
    bad = tok.clone()
    bad[[0, 5, 19]] = torch.tensor([-1, V, 2 ** 31 - 1], dtype=torch.int32, device="cuda")
    (lp, H, lse), _ = _decode(h, W, tok, 1.0)
    (lp2, H2, lse2), _ = _decode(h, W, bad, 1.0)
    assert torch.isnan(lp2[[0, 5, 19]]).all()
    ok = [i for i in range(T) if i not in (0, 5, 19)]
    assert bits_equal(lp2[ok], lp[ok])
    assert bits_equal(H2, H) and bits_equal(lse2, lse)


def test_partials_merge_equal_halves():
    """The two-stage calls (whole-tile partials) give the decode call's bits."""
    T, d, V = 48, 256, 4096 + 200
    h, W = inputs(T, d, V, seed=44)
    tok = _tokens(T, V, seed=44)
    ws = torch.empty(tim.workspace_size(T, d, V, Mode.ROLLOUT), dtype=torch.uint8, device="cuda")
    tim.logprobs_partials(h, W, tok, ws, 1.3, mode=Mode.ROLLOUT)
    staged = tim.logprobs_merge(ws, tok, V)
    direct = tim.logprobs(h, W, tok, 1.3, mode=Mode.ROLLOUT, lse=True)
    _same(staged, direct)


def test_halves_uniform_rows_closed_form():
    """h = 0: every logit is 0, logp = -log V and H = log V, in a decode batch."""
    T, d, V = 64, 256, 151936
    h = torch.zeros(T, d, dtype=torch.bfloat16, device="cuda")
    _, W = inputs(1, d, V, seed=45)
    tok = _tokens(T, V, seed=45)
    (lp, H, _), _ = _decode(h, W, tok, 1.0)
    check_close("uniform logp", lp, np.full(T, -np.log(V)), 2e-5)
    check_close("uniform entropy", H, np.full(T, np.log(V)), 2e-5)


@pytest.mark.parametrize("V", [32768 + 1, 65536 + 300, 151936, 300000, 2048 * 256])
def test_quad_merge_equals_wave_merge(V):
    """Launches of at most 512 rows merge with four waves per row (quarters of
    the leaves, then (q0 + q1) + (q2 + q3)); larger ones with one wave per row.
    Both are the same balanced tree: merging the first rows' partials alone
    gives the bits of merging them within a larger launch."""
    T, d = 600, 128
    print(f"case quad merge V={V}", flush=True)
    h, W = inputs(T, d, V, seed=V % 977)
    tok = random_tokens(T, V, seed=V % 977)
    ws = torch.empty(tim.workspace_size(T, d, V, Mode.TRAINING), dtype=torch.uint8, device="cuda")
    tim.logprobs_partials(h, W, tok, ws, 1.0, mode=Mode.TRAINING)
    wave = tim.logprobs_merge(ws, tok, V)                      # 600 rows: one wave per row
    for n in (1, 100, 512):
        quad = tim.logprobs_merge(ws, tok[:n].contiguous(), V)    # four waves per row
        for x, y in zip(quad, wave):
            assert bits_equal(x, y[:n])


def test_decode_128_row_tiles_full_size():
    """d = 4096, V = 151936, decode batches of 65..128 rows (the 128-row half
    tiles of four waves): bitwise equal to the training path, and to the
    oracle on sampled rows."""
    T, d, V = 128, 4096, 151936
    h, W = inputs(T, d, V, seed=46, w_std=0.02)
    tok = _tokens(T, V, seed=46)
    trn = tim.logprobs(h, W, tok, 1.0, mode=Mode.TRAINING, lse=True)
    for n in (65, 100, 128):
        dec, per_row = _decode(h[:n].contiguous(), W, tok[:n].contiguous(), 1.0)
        assert per_row == _per_row(V, n)
        for x, y in zip(dec, trn):
            assert bits_equal(x, y[:n])
    rows = [0, 1, 63, 64, 65, 99, 127]
    ref_lp, ref_H = oracle_rows(h, W, tok, 1.0, rows=rows)
    check_close("decode-128 logp", trn[0], ref_lp, TOL_LOGP, rows=rows)
    check_close("decode-128 entropy", trn[1], ref_H, TOL_ENT, rows=rows)


@pytest.mark.parametrize("d", [128, 384, 640])
@pytest.mark.parametrize("V", [1, 129, 383, 4096 + 77, 4096 + 200])
@pytest.mark.parametrize("T", [65, 96, 97, 127, 128])
def test_decode_65_128_bitwise_equal_training(d, V, T):
    """Decode batches of 65..128 rows (half tiles of 128 rows, four row waves
    of 32, some of them empty or cut by the batch) at hidden sizes of 2, 6 and
    10 stages and every kind of vocabulary tail, each call repeated: bitwise equal
    to the training path, and within tolerance of the oracle at d = 128."""
    print(f"case decode 65..128 d={d} V={V} T={T}", flush=True)
    h, W = inputs(T, d, V, seed=(V + 5 * T + d) % 1000, w_std=0.1)
    tok = _tokens(T, V, seed=V + 3 * T + d)
    trn = tim.logprobs(h, W, tok, 0.7, mode=Mode.TRAINING, lse=True)
    for _ in range(2):
        dec, per_row = _decode(h, W, tok, 0.7)
        assert per_row == -(-V // 128)
        _same(dec, trn)
    if d == 128:
        ref_lp, ref_H = oracle_rows(h, W, tok, 0.7)
        check_close(f"decode 65..128 logp d={d} V={V}", dec[0], ref_lp, TOL_LOGP)
        check_close(f"decode 65..128 entropy d={d} V={V}", dec[1], ref_H, TOL_ENT)


@pytest.mark.parametrize("d", [128, 256, 384, 640])
@pytest.mark.parametrize("V", [1, 129, 383, 4096 + 77, 4096 + 200, 600 * 256])
@pytest.mark.parametrize("T", [129, 160, 193, 255, 256])
def test_decode_129_256_bitwise_equal_training(d, V, T):
    """Decode batches of 129..256 rows (whole tiles, one 256-row tile,
    persistent): hidden sizes of 2 .. 10 stages, row tiles cut by the batch,
    every kind of vocabulary tail. Bitwise equal to the training path, and
    within tolerance of the oracle at small V."""
    print(f"case decode 129..256 d={d} V={V} T={T}", flush=True)
    h, W = inputs(T, d, V, seed=(V + 7 * T + d) % 1000, w_std=0.1)
    tok = _tokens(T, V, seed=V + T + d)
    dec, per_row = _decode(h, W, tok, 0.7)
    assert per_row == -(-V // 256)
    trn = tim.logprobs(h, W, tok, 0.7, mode=Mode.TRAINING, lse=True)
    _same(dec, trn)
    if V <= 4096 + 200 and d <= 256:
        ref_lp, ref_H = oracle_rows(h, W, tok, 0.7)
        check_close(f"decode 129..256 logp d={d} V={V}", dec[0], ref_lp, TOL_LOGP)
        check_close(f"decode 129..256 entropy d={d} V={V}", dec[1], ref_H, TOL_ENT)


def test_decode_129_256_full_size():
    """d = 4096, V = 151936, decode batches of 129..256 rows (several tiles per
    workgroup): bitwise equal to the training path, and to the oracle on
    sampled rows of every row wave."""
    T, d, V = 256, 4096, 151936
    h, W = inputs(T, d, V, seed=47, w_std=0.02)
    tok = _tokens(T, V, seed=47)
    trn = tim.logprobs(h, W, tok, 1.0, mode=Mode.TRAINING, lse=True)
    for n in (129, 200, 256):
        dec, per_row = _decode(h[:n].contiguous(), W, tok[:n].contiguous(), 1.0)
        assert per_row == 594
        for x, y in zip(dec, trn):
            assert bits_equal(x, y[:n])
    rows = [0, 1, 31, 32, 100, 128, 129, 160, 199, 224, 255]
    ref_lp, ref_H = oracle_rows(h, W, tok, 1.0, rows=rows)
    check_close("decode 129..256 logp", trn[0], ref_lp, TOL_LOGP, rows=rows)
    check_close("decode 129..256 entropy", trn[1], ref_H, TOL_ENT, rows=rows)


def test_decode_repeated_calls_identical():
    """Repeated decode calls of 129..224 rows (row waves of the 256-row tile
    with no rows) at several hidden sizes return the same bits every time, and
    those of the training path."""
    V = 4096 + 200
    for d in (256, 384, 640):
        for T in (129, 160, 193):
            print(f"case repeated d={d} T={T}", flush=True)
            h, W = inputs(T, d, V, seed=T + d, w_std=0.1)
            tok = _tokens(T, V, seed=T + d)
            trn = tim.logprobs(h, W, tok, 0.7, mode=Mode.TRAINING, lse=True)
            for _ in range(4):
                dec, _ = _decode(h, W, tok, 0.7)
                _same(dec, trn)
