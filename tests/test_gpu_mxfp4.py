"""GPU parity of the MXFP4 cast path (Sec. 4.8 Cast, Sec. 6.4: the
reconstruction fed to MXFP4, OCP Microscaling blocks of 32 with E8M0 scales
and E2M1 elements) against the oracle: the decoded code nibbles and block
scale bytes of g c bit for bit, the activation prep's nibbles and scales bit
for bit, and the block-scaled GEMM on the gfx950 scaled matrix cores within
1e-4 of max(|ref|, rms(ref)): the products of two E2M1 values times a power
of two are exact in fp32, and only the fp32 sums across blocks round."""
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


def pack_nibbles(codes):
    """Two E2M1 codes per byte, the even k in the low nibble."""
    c = np.asarray(codes, dtype=np.uint8)
    return (c[:, 0::2] | (c[:, 1::2] << 4)).astype(np.uint8)


@pytest.mark.parametrize("lat", [O.E8, O.D4, O.Z])
def test_decode_mxfp4_codes_and_scales(hq, lat):
    snr = PT.op_snr("E8", 4.0) if lat == O.E8 else 30.0
    P = PT.oracle_params(lat, snr, rht_seed=29)
    x = gauss(40, 1024, 35, 0.02, torch.bfloat16)
    x[:, 7::97] *= 8  # a few large codes: their blocks' small codes round to 0
    x[3, :] = 0.0     # an all-zero row: every block takes X = -127
    print(f"[parity] decode_mxfp4 {LAT_NAMES[lat]}", flush=True)
    plan, s = encode_gpu(hq, P, snr, x)
    codes, scales = hq.hq_decode_mxfp4(plan, s)
    torch.cuda.synchronize()
    oc, norms, _, _ = O.frontend(P, x.float().numpy())
    o4, os_ = O.weight_codes_mxfp4(oc, O.weight_factors(P, norms, 40, 1024), 128)
    assert np.array_equal(scales.cpu().numpy(), os_)
    assert np.array_equal(codes.cpu().numpy(), pack_nibbles(o4))
    assert (os_[3] == 0).all()
    # a row range decodes the same bytes as the whole matrix's rows
    c2, s2 = hq.hq_decode_mxfp4(plan, s, row0=9, rows=13)
    torch.cuda.synchronize()
    assert torch.equal(c2.cpu(), codes[9:22].cpu())
    assert torch.equal(s2.cpu(), scales[9:22].cpu())


def test_act_prep_mxfp4(hq):
    from paper_2606_23406_amd import workloads
    a = workloads.activations(tokens=64, features=1024)
    a[5] = 0.0  # an all-zero token
    a[9, :300] *= 1e-6  # blocks far below the row's others
    P = PT.oracle_params(O.E8, 20.0, rht_seed=47)
    plan = PT.gpu_plan(hq, P, 20.0, 1024)
    print("[parity] act_prep_mxfp4 64x1024", flush=True)
    xq, xs = hq.hq_act_prep_mxfp4(plan, a.cuda())
    torch.cuda.synchronize()
    o4, os_ = O.act_prep_mxfp4(a.float().numpy(), 128, 47)
    assert np.array_equal(xs.cpu().numpy(), os_)
    assert np.array_equal(xq.cpu().numpy(), pack_nibbles(o4))


@pytest.mark.parametrize("M,N,K", [(128, 256, 1024), (200, 384, 1024), (64, 96, 512),
                                   (300, 160, 2560), (70, 100, 512)])
def test_gemm_mxfp4_blockscaled(hq, M, N, K):
    from paper_2606_23406_amd import workloads
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=59)
    w = gauss(N, K, 67, 0.02, torch.bfloat16)
    a = workloads.activations(tokens=M, features=K)
    print(f"[parity] gemm mxfp4 M={M} N={N} K={K}", flush=True)
    plan, s = encode_gpu(hq, P, snr, w)
    codes, ws = hq.hq_decode_mxfp4(plan, s)
    xq, xs = hq.hq_act_prep_mxfp4(plan, a.cuda())
    out32 = hq.hq_gemm_mxfp4_blockscaled(plan, xq, xs, codes, ws, out_dtype=torch.float32)
    out16 = hq.hq_gemm_mxfp4_blockscaled(plan, xq, xs, codes, ws, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    oc, norms, _, _ = O.frontend(P, w.float().numpy())
    og = O.weight_factors(P, norms, N, K)
    o4, ows = O.weight_codes_mxfp4(oc, og, 128)
    ox4, oxs = O.act_prep_mxfp4(a.float().numpy(), 128, 59)
    # the GPU's operands are the oracle's, byte for byte, before the product
    assert np.array_equal(codes.cpu().numpy(), pack_nibbles(o4))
    assert np.array_equal(ws.cpu().numpy(), ows)
    assert np.array_equal(xq.cpu().numpy(), pack_nibbles(ox4))
    ref = O.gemm_mxfp4(o4, ows, ox4, oxs)
    got = out32.cpu().numpy().astype(np.float64)
    denom = np.maximum(np.abs(ref), np.sqrt((ref ** 2).mean()))
    err = float(np.max(np.abs(got - ref) / denom))
    print(f"[parity] gemm mxfp4 M={M} N={N} K={K}: worst error {err:.2e}", flush=True)
    assert err <= 1e-4
    assert torch.equal(out16.cpu(), out32.cpu().to(torch.bfloat16))
    # and it approximates the int8 path's product (both cast the same decode)
    ref8 = O.gemm_blockscaled(oc, og, *O.act_prep(a.float().numpy(), 128, 59), 128)
    rel = np.linalg.norm(got - ref8) / np.linalg.norm(ref8)
    print(f"[parity] gemm mxfp4 vs int8 path: relative difference {rel:.3f}", flush=True)
    assert rel < 0.35

