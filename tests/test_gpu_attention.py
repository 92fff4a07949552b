"""GPU parity of hq_decode_attention (one query token per sequence over coded
K and V streams) against the oracle's attention over the decoded rows.

Both streams are encoded on the GPU, KV-style (signs rotation, dither, fp16
norms, appended in chunks); the oracle attends over the rows that the
stream's own codes decode to.  Bar: every output within 2e-5 of the largest
|v^| among the sequence's value rows (fp32 sums; the largest error seen,
3e-7, is some 60x smaller), the bf16 output the fp32 one rounded to nearest
even."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from tests import parity as PT

pytestmark = pytest.mark.gpu

LAT_NAMES = {O.E8: "E8", O.D4: "D4", O.A2: "A2", O.Z: "Z"}
SNR = {O.E8: PT.op_snr("E8", 2.0), O.D4: 12.0, O.A2: PT.op_snr("A2", 1.7), O.Z: PT.op_snr("Z", 1.7)}
N = 128
INVALID_ARG = -1 & 0xFFFFFFFF


@pytest.fixture(scope="module")
def hq():
    from paper_2606_23406_amd import hq as H
    H.lib()
    assert torch.cuda.is_available()
    return H


def coded(hq, P, x, chunk=16):
    """x encoded on the GPU in appended chunks; returns plan, stream and the
    stream's own codes and norms (oracle-parsed where they differ)."""
    rows, cols = x.shape
    plan = PT.gpu_plan(hq, P, SNR[P.lattice], cols)
    s = hq.EncodedStream(plan, rows)
    xd = x.cuda()
    for r0 in range(0, rows, chunk):
        hq.hq_encode(plan, xd[r0:r0 + chunk], s, append=r0 > 0)
    torch.cuda.synchronize()
    res = PT.compare_streams(P, x.float().numpy(), PT.gpu_stream_arrays(s, rows))
    codes = res["codes"] if res["gpu_codes"] is None else res["gpu_codes"]
    return plan, s, codes, res["norms"]


def kv_pair(hq, lat, rows, hkv, seed, kv=True):
    g = torch.Generator().manual_seed(seed)
    k = torch.randn((rows, hkv * N), generator=g)
    k[:, 3::N] *= 10  # outlier channels
    v = torch.randn((rows, hkv * N), generator=g)
    k, v = k.to(torch.bfloat16), v.to(torch.bfloat16)
    opts = dict(rotation=1, dither=True, norm_fp16=True) if kv else {}
    pk = PT.oracle_params(lat, SNR[lat], rht_seed=41, rot_seed=42, dither_seed=43 + lat, **opts)
    pv = PT.oracle_params(lat, SNR[lat], rht_seed=51, rot_seed=52, dither_seed=53 + lat, **opts)
    return (pk,) + coded(hq, pk, k), (pv,) + coded(hq, pv, v)


def check(hq, K, V, q, table, lens, bt, label, scale=N ** -0.5, wk=None, wv=None):
    pk, plk, sk, kc, kn = K
    pv, plv, sv, vc, vn = V
    W = 0 if wk is None else wk.shape[1]
    ref = O.decode_attention(pk, kc, kn, pv, vc, vn, q.float().numpy(), table, lens, bt, scale,
                             window=W, window_k=None if wk is None else wk.float().numpy(),
                             window_v=None if wv is None else wv.float().numpy())
    vd = O.backend(pv, vc, vn)
    B, Hq = q.shape[0], q.shape[1]
    G = Hq // (vd.shape[1] // N)
    tab, ln = torch.from_numpy(table).cuda(), torch.from_numpy(np.asarray(lens, np.int32)).cuda()
    print(f"[attn] {label} q={q.dtype} batch={B} heads={Hq} lens={list(lens)}", flush=True)
    win = {} if wk is None else dict(window_k=wk.cuda(), window_v=wv.cuda())
    out = hq.hq_decode_attention(plk, sk, plv, sv, q.cuda(), tab, ln, bt, scale=scale, **win)
    out16 = hq.hq_decode_attention(plk, sk, plv, sv, q.cuda(), tab, ln, bt, scale=scale,
                                   out_dtype=torch.bfloat16, **win)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    worst = 0.0
    for b in range(B):
        t = np.arange(lens[b])
        rows = table[b][t // bt].astype(np.int64) * bt + t % bt
        w = min(W, lens[b])
        rows = rows[:lens[b] - w]
        for h in range(Hq):
            cs = slice((h // G) * N, (h // G + 1) * N)
            vals = np.abs(vd[rows, cs])
            if w:
                vals = np.concatenate([vals, np.abs(wv.float().numpy()[b, :, cs])])
            unit = vals.max() if lens[b] else 1.0
            err = np.abs(got[b, h] - ref[b, h]).max() / unit
            worst = max(worst, err)
            assert err <= 2e-5, (label, b, h, err)
    assert torch.equal(out16.cpu(), out.cpu().to(torch.bfloat16))
    st = sk.read_stats()
    assert st["status"] == 0 and st["corrupt_substreams"] == 0, st
    print(f"[attn] {label}: worst error {worst:.2e} of max |v|", flush=True)
    return got


def paged(rng, lens, bt, nblocks):
    """A block table giving each sequence distinct blocks in shuffled order."""
    need = [-(-n // bt) for n in lens]
    width = max(1, max(need))
    perm = rng.permutation(nblocks)
    assert sum(need) <= nblocks
    table = np.zeros((len(lens), width), dtype=np.int32)
    i = 0
    for b, k in enumerate(need):
        table[b, :k] = perm[i:i + k]
        i += k
    return table


@pytest.mark.parametrize("lat", [O.E8, O.D4, O.A2, O.Z])
def test_attention_kv_streams(hq, lat):
    # 4 KV heads (one sub-stream per row), 2 query heads each; ragged lengths
    # over a shuffled paged cache of 16-token blocks, one sequence empty
    rng = np.random.default_rng(60 + lat)
    K, V = kv_pair(hq, lat, 40 * 16, 4, 70 + lat)
    lens = [37, 1, 0, 300, 16]
    table = paged(rng, lens, 16, 40)
    for qdt in (torch.float32, torch.bfloat16):
        q = torch.from_numpy(rng.standard_normal((5, 8, N)).astype(np.float32)).to(qdt)
        check(hq, K, V, q, table, lens, 16, f"kv {LAT_NAMES[lat]}")


@pytest.mark.parametrize("group", [1, 4, 8])
def test_attention_head_groups_and_splits(hq, group):
    # 8 KV heads (two sub-streams per row), 1 / 4 / 8 query heads each; one
    # long sequence spans many token splits
    rng = np.random.default_rng(80 + group)
    K, V = kv_pair(hq, O.E8, 2400, 8, 90)
    lens = [2000, 3, 290]
    table = paged(rng, lens, 16, 2400 // 16)
    q = torch.from_numpy(rng.standard_normal((3, 8 * group, N)).astype(np.float32))
    check(hq, K, V, q, table, lens, 16, f"E8 group {group}")


@pytest.mark.parametrize("W", [8, 32])
def test_attention_residual_window(hq, W):
    # the last min(W, len) tokens read exact from a ring (token t in slot
    # t % W), bf16 and fp32 rings; lengths below, at and above W, and empty
    rng = np.random.default_rng(95 + W)
    K, V = kv_pair(hq, O.E8, 40 * 16, 4, 96)
    lens = [37, 5, 0, W, 300]
    table = paged(rng, lens, 16, 40)
    q = torch.from_numpy(rng.standard_normal((5, 8, N)).astype(np.float32))
    for dt in (torch.bfloat16, torch.float32):
        wk = torch.from_numpy(rng.standard_normal((5, W, 4 * N)).astype(np.float32)).to(dt)
        wk[:, :, 3::N] *= 10
        wv = torch.from_numpy(rng.standard_normal((5, W, 4 * N)).astype(np.float32)).to(dt)
        check(hq, K, V, q, table, lens, 16, f"E8 window {W} {dt}", wk=wk, wv=wv)


def test_attention_plain_streams_and_contiguous_table(hq):
    # weight-style plans (no rotation, dither or fp16 norms) and one block per
    # sequence (a contiguous cache)
    rng = np.random.default_rng(7)
    K, V = kv_pair(hq, O.D4, 300, 4, 8, kv=False)
    table = np.array([[0], [1]], dtype=np.int32)
    lens = [150, 97]
    q = torch.from_numpy(rng.standard_normal((2, 4, N)).astype(np.float32))
    check(hq, K, V, q, table, lens, 150, "D4 plain, contiguous", scale=0.2)


def test_attention_repeats_bit_for_bit(hq):
    rng = np.random.default_rng(9)
    K, V = kv_pair(hq, O.A2, 640, 4, 10)
    lens = [500, 77]
    table = torch.from_numpy(paged(rng, lens, 16, 40)).cuda()
    ln = torch.tensor(lens, dtype=torch.int32, device="cuda")
    q = torch.randn((2, 16, N), device="cuda")
    a = hq.hq_decode_attention(K[1], K[2], V[1], V[2], q, table, ln, 16)
    b = hq.hq_decode_attention(K[1], K[2], V[1], V[2], q, table, ln, 16)
    assert torch.equal(a, b)


def test_attention_errors(hq):
    rng = np.random.default_rng(12)
    K, V = kv_pair(hq, O.E8, 64, 4, 13)
    plk, sk, plv, sv = K[1], K[2], V[1], V[2]
    table = torch.tensor([[0, 1, 2, 3]], dtype=torch.int32, device="cuda")
    ln = torch.tensor([64], dtype=torch.int32, device="cuda")
    q = torch.randn((1, 8, N), device="cuda")
    with pytest.raises(hq.HQError):  # 12 query heads over 4 KV heads
        hq.hq_decode_attention(plk, sk, plv, sv, torch.randn((1, 12, N), device="cuda"), table, ln, 16)
    with pytest.raises(hq.HQError):  # workspace too small
        hq.hq_decode_attention(plk, sk, plv, sv, q, table, ln, 16,
                               workspace=torch.empty(64, dtype=torch.uint8, device="cuda"))
    other = hq.hq_plan(128, hq.HQ_E8, 0.0, 5, -1, 1024, snr_db=20.0)
    with pytest.raises(hq.HQError):  # key and value plans of different widths
        hq.hq_decode_attention(plk, sk, other, sv, q, table, ln, 16)
    big = torch.zeros((1, 257, 4 * N), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(hq.HQError):  # residual window above 256 tokens
        hq.hq_decode_attention(plk, sk, plv, sv, q, table, ln, 16, window_k=big, window_v=big)
    # a block id past the streams' rows is skipped and reported; the rest is
    # the attention over the remaining tokens
    sk.reset_stats()
    bad = torch.tensor([[0, 1, 2, 1000]], dtype=torch.int32, device="cuda")
    out = hq.hq_decode_attention(plk, sk, plv, sv, q, bad, ln, 16)
    torch.cuda.synchronize()
    assert sk.read_stats()["status"] == INVALID_ARG
    ref = hq.hq_decode_attention(plk, sk, plv, sv, q, table, torch.tensor([48], dtype=torch.int32,
                                                                           device="cuda"), 16)
    torch.testing.assert_close(out, ref, rtol=0, atol=1e-5)
    # a length past the table is clamped and reported
    sk.reset_stats()
    hq.hq_decode_attention(plk, sk, plv, sv, q, table, torch.tensor([65], dtype=torch.int32,
                                                                    device="cuda"), 16)
    torch.cuda.synchronize()
    assert sk.read_stats()["status"] == INVALID_ARG
