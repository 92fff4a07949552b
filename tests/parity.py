"""Parity helpers: run the HIP path through the C ABI and the oracle on the same
inputs, and compare what the method fixes (test infrastructure)."""
import json
import os

import numpy as np
import torch

from oracle import oracle as O

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
MARGIN_EXEMPT = 1e-6


def op_snr(name, bps):
    pts = json.load(open(os.path.join(GOLDEN, "operating_points.json")))["points"]
    for p in pts:
        if p["lattice"] == name and abs(p["bps"] - bps) < 1e-9:
            return p["snr_db"]
    raise KeyError((name, bps))


def oracle_params(lat, snr, rht_seed=0, rice_k=-1, rotation=0, rot_seed=0, dither=False,
                  dither_seed=0, norm_fp16=False, qjl=None, tile=128, substream=512):
    return O.Params(tile=tile, lattice=lat, alpha=O.alpha(lat, snr), substream=substream, rice_k=rice_k,
                    norm_fp16=norm_fp16, rht_seed=rht_seed, rotation=rotation, dither=dither,
                    rot_seed=rot_seed, dither_seed=dither_seed, qjl=qjl)


def gpu_plan(hq, P: O.Params, snr, cols):
    plan = hq.hq_plan(P.tile, P.lattice, 0.0, P.rht_seed, P.rice_k, cols, rotation=P.rotation,
                      dither=P.dither, rot_seed=P.rot_seed, dither_seed=P.dither_seed,
                      norm_fp16=P.norm_fp16, snr_db=snr, qjl=P.qjl,
                      substream=0 if P.substream == 512 else P.substream)
    assert np.float32(plan.info.alpha) == np.float32(P.alpha), "alpha differs from the oracle's"
    return plan


def gpu_stream_arrays(s, rows):
    spr = s.plan.info.subs_per_row
    nsub = rows * spr
    offsets = s.offsets[: nsub + 1].cpu().numpy().view(np.uint32).copy()
    end = int(offsets[-1])
    payload = s.payload[:end].cpu().numpy().view(np.uint32).copy()
    kparam = s.kparam[:nsub].cpu().numpy().copy()
    tpr = s.plan.info.tiles_per_row
    norms = s.norms[: rows * tpr].cpu()
    norms = (norms.numpy().view(np.uint16) if norms.dtype == torch.float16 else norms.numpy())
    return payload, offsets, kparam, norms.reshape(rows, tpr).copy()


def compare_streams(P: O.Params, x_np, gpu, row0=0, check_decode=None):
    """Compare a GPU-encoded stream (payload, offsets, kparam, norms arrays for
    rows row0.. of a stream) with the oracle on the same rows.  Returns a dict
    of counts; raises AssertionError on any non-exempt difference."""
    g_pay, g_off, g_kp, g_norm = gpu
    rows, cols = x_np.shape
    codes, norms, zin, _ = O.frontend(P, x_np, row0=row0, want_z=True)
    o_pay, o_off, o_kp, bits = O.pack(P, codes, row0=0)
    S = P.substream
    o_off = o_off[: rows * (cols // S) + 1]
    o_kp = o_kp[: rows * (cols // S)]
    assert np.array_equal(g_norm.view(np.uint8), norms.view(np.uint8)), "stored norms differ"
    m = O.DIM[P.lattice]
    gsz = np.diff(g_off.astype(np.int64))
    osz = np.diff(o_off.astype(np.int64))
    nsub = osz.size
    exempt_blocks = 0
    exempt_subs = 0
    mismatched = []
    for s in range(nsub):
        gw = g_pay[g_off[s] - g_off[0]: g_off[s + 1] - g_off[0]]
        ow = o_pay[o_off[s]: o_off[s + 1]]
        if g_kp[s] == o_kp[s] and gsz[s] == osz[s] and np.array_equal(gw, ow):
            continue
        mismatched.append(s)
    g_codes = None
    if mismatched:
        # decode the GPU stream with the oracle's unpacker to get its codes
        rel_off = (g_off.astype(np.int64) - int(g_off[0])).astype(np.uint32)
        g_codes, rc = O.unpack(P, g_pay, rel_off, g_kp, rows, cols, 0)
        assert rc == O.OK, "GPU stream does not parse"
        flat_z = zin.reshape(-1, m)
        flat_c = codes.reshape(-1, m)
        flat_g = g_codes.reshape(-1, m)
        for s in mismatched:
            b0, b1 = s * S // m, (s + 1) * S // m
            diff = np.any(flat_c[b0:b1] != flat_g[b0:b1], axis=1)
            if not diff.any():
                raise AssertionError(f"sub-stream {s}: same codes, different bits")
            mg = O.margins(P.lattice, flat_z[b0:b1][diff], flat_c[b0:b1][diff])
            if np.any(mg >= MARGIN_EXEMPT):
                bad = np.nonzero(diff)[0][mg >= MARGIN_EXEMPT]
                raise AssertionError(f"sub-stream {s}: codes differ at blocks {bad[:8]} with "
                                     f"margins {mg[mg >= MARGIN_EXEMPT][:8]}")
            exempt_blocks += int(diff.sum())
            exempt_subs += 1
            # the GPU's bits must be exactly the oracle's Rice code of the GPU's symbols
            rp, roff, rkp, _ = O.pack(P, g_codes[(s * S) // cols:(s * S) // cols + 1], row0=0)
            srow = s % (cols // S)
            gw = g_pay[g_off[s] - g_off[0]: g_off[s + 1] - g_off[0]]
            assert rkp[srow] == g_kp[s]
            assert np.array_equal(rp[roff[srow]:roff[srow + 1]], gw)
    return {"substreams": nsub, "exempt_substreams": exempt_subs, "exempt_blocks": exempt_blocks,
            "payload_bits": bits, "codes": codes, "gpu_codes": g_codes, "norms": norms,
            "mismatched": mismatched}


def tiles_with_code_diffs(codes, g_codes, tile=128):
    if g_codes is None:
        return np.zeros(codes.shape[0] * codes.shape[1] // tile, dtype=bool)
    d = (codes != g_codes).reshape(-1, tile)
    return d.any(axis=1)


def lattice_unit(P: O.Params, norms):
    """u = r_s / (alpha sqrt(n)) per tile (the lattice step in input units)."""
    r = O.f16_bits_to_f32(norms) if P.norm_fp16 else norms.reshape(-1).astype(np.float32)
    return r.astype(np.float64) / (float(P.alpha) * np.sqrt(P.tile))
