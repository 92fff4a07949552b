"""GPU parity of the fp8 cast path (Sec. 4.8 / 6.3: OCP E4M3 at the
matrix-core boundary) against the oracle: the decoded E4M3 code bytes and
tile factors bit for bit, the activation prep's bytes and scales bit for bit,
and the block-scaled GEMM on the fp8 matrix cores within 1e-4 of
max(|ref|, rms(ref)) (E4M3 products are exact in fp32; the largest error
seen, 3e-5, is the fp32 tile sums' rounding), its bf16 output the fp32 one
rounded to nearest even."""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from tests import parity as PT
from tests.test_gpu_parity import encode_gpu, gauss

pytestmark = pytest.mark.gpu

LAT_NAMES = {O.E8: "E8", O.D4: "D4", O.Z: "Z"}


@pytest.fixture(scope="module")
def hq():
    from paper_2606_23406_amd import hq as H
    H.lib()
    assert torch.cuda.is_available()
    return H


@pytest.mark.parametrize("lat", [O.E8, O.D4, O.Z])
def test_decode_fp8_codes_and_factors(hq, lat):
    snr = PT.op_snr("E8", 4.0) if lat == O.E8 else 30.0
    P = PT.oracle_params(lat, snr, rht_seed=23)
    x = gauss(40, 1024, 33, 0.02, torch.bfloat16)
    x[:, 7::97] *= 8  # some large codes (beyond 16: the cast rounds them)
    print(f"[parity] decode_fp8 {LAT_NAMES[lat]}", flush=True)
    plan, s = encode_gpu(hq, P, snr, x)
    codes, g = hq.hq_decode_fp8(plan, s)
    torch.cuda.synchronize()
    oc, norms, _, _ = O.frontend(P, x.float().numpy())
    assert np.abs(oc).max() > 16
    assert np.array_equal(codes.cpu().numpy(), O.weight_codes_fp8(oc))
    assert np.array_equal(g.cpu().numpy(), O.weight_factors(P, norms, 40, 1024))


def test_act_prep_fp8(hq):
    from paper_2606_23406_amd import workloads
    a = workloads.activations(tokens=64, features=1024)
    P = PT.oracle_params(O.E8, 20.0, rht_seed=43)
    plan = PT.gpu_plan(hq, P, 20.0, 1024)
    print("[parity] act_prep_fp8 64x1024", flush=True)
    xq, sx = hq.hq_act_prep_fp8(plan, a.cuda())
    torch.cuda.synchronize()
    oxq, osx = O.act_prep_fp8(a.float().numpy(), 128, 43)
    assert np.array_equal(sx.cpu().numpy(), osx)
    assert np.array_equal(xq.cpu().numpy(), oxq)


@pytest.mark.parametrize("M,N,K", [(128, 256, 1024), (200, 384, 1024), (64, 96, 1024),
                                   (300, 200, 512), (40, 136, 2560), (70, 100, 512)])
def test_gemm_fp8_blockscaled(hq, M, N, K):
    # K = 512: four stages (the shortest K a plan takes); 2560: twenty, the LDS ring wrapping;
    # N = 100: bf16 output rows of 200 bytes, every other one off 16-byte alignment (element stores)
    from paper_2606_23406_amd import workloads
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=53)
    w = gauss(N, K, 63, 0.02, torch.bfloat16)
    a = workloads.activations(tokens=M, features=K)
    print(f"[parity] gemm fp8 M={M} N={N} K={K}", flush=True)
    plan, s = encode_gpu(hq, P, snr, w)
    codes, g = hq.hq_decode_fp8(plan, s)
    xq, sx = hq.hq_act_prep_fp8(plan, a.cuda())
    out32 = hq.hq_gemm_fp8_blockscaled(plan, xq, sx, codes, g, out_dtype=torch.float32)
    out16 = hq.hq_gemm_fp8_blockscaled(plan, xq, sx, codes, g, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    oc, norms, _, _ = O.frontend(P, w.float().numpy())
    og = O.weight_factors(P, norms, N, K)
    oxq, osx = O.act_prep_fp8(a.float().numpy(), 128, 53)
    ref = O.gemm_fp8_blockscaled(O.weight_codes_fp8(oc), og, oxq, osx, 128)
    got = out32.cpu().numpy().astype(np.float64)
    denom = np.maximum(np.abs(ref), np.sqrt((ref ** 2).mean()))
    err = float(np.max(np.abs(got - ref) / denom))
    print(f"[parity] gemm fp8 M={M} N={N} K={K}: worst error {err:.2e}", flush=True)
    assert err <= 1e-4
    # bf16 output: the fp32 one rounded to nearest even (the fp32 tile sums
    # round, unlike the int8 path's exact int32 ones)
    assert torch.equal(out16.cpu(), out32.cpu().to(torch.bfloat16))
    # and it approximates the int8 path's product (both cast the same decode)
    ref8 = O.gemm_blockscaled(oc, og, *O.act_prep(a.float().numpy(), 128, 53), 128)
    assert np.linalg.norm(got - ref8) / np.linalg.norm(ref8) < 0.1
