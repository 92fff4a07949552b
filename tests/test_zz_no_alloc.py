"""hq_encode_noalloc (the encode entry point that allocates nothing, with
the library's fixed look-back scratch) against hq_encode, through the C ABI:
the same payload, offsets, k bytes, norms and stats, on calls in a row whose
second is smaller, at the scratch's largest size, and with appends; sizes past
the scratch are rejected before any work is enqueued."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def hq():
    from paper_2606_23406_amd import hq as H
    H.lib()
    assert torch.cuda.is_available()
    return H


def same_stream(a, b, rows):
    spr = a.plan.info.subs_per_row
    nsub = rows * spr
    assert a.rows == b.rows == rows
    assert torch.equal(a.offsets[:nsub + 1], b.offsets[:nsub + 1])
    end = int(a.offsets[nsub].item()) & 0xFFFFFFFF
    assert torch.equal(a.payload[:end], b.payload[:end])
    assert torch.equal(a.kparam[:nsub], b.kparam[:nsub])
    tpr = a.plan.info.tiles_per_row
    assert torch.equal(a.norms[:rows * tpr].view(torch.int16 if a.norms.dtype == torch.float16
                                                else torch.int32),
                       b.norms[:rows * tpr].view(torch.int16 if b.norms.dtype == torch.float16
                                                else torch.int32))
    sa, sb = a.read_stats(), b.read_stats()
    assert sa == sb and sa["status"] == 0, (sa, sb)
    return end


def bf16_rows(rows, cols, seed, scale=0.02):
    g = torch.Generator(device="cuda").manual_seed(seed)
    return (torch.randn((rows, cols), generator=g, device="cuda") * scale).to(torch.bfloat16)


def test_noalloc_matches_encode_two_calls(hq):
    """Call 1 fills 2100 x 4096 (the four-sub-streams-per-wave shape), call 2
    a smaller 300 x 4096 (one per wave): each equals hq_encode's stream."""
    plan = hq.hq_plan(128, hq.HQ_E8, 4.0, 7, -1, 4096)
    for rows, seed in ((2100, 1), (300, 2)):
        print(f"[noalloc] E8@4 {rows}x4096", flush=True)
        x = bf16_rows(rows, 4096, seed)
        ref = hq.EncodedStream(plan, rows)
        got = hq.EncodedStream(plan, rows)
        hq.hq_encode(plan, x, ref)
        hq.hq_encode_noalloc(plan, x, got)
        torch.cuda.synchronize()
        assert same_stream(ref, got, rows) > 0


def test_noalloc_kv_appends(hq):
    """KV quantize-on-append (signs + dither + fp16 norms): three appends,
    the later ones smaller, each continuing the stream as hq_encode does."""
    plan = hq.hq_plan(128, hq.HQ_E8, 2.0, 3, -1, 1024, rotation=hq.HQ_ROT_SIGNS, dither=True,
                      rot_seed=5, dither_seed=77, norm_fp16=True)
    total = 0
    ref = hq.EncodedStream(plan, 4096)
    got = hq.EncodedStream(plan, 4096)
    for rows, seed in ((2048, 3), (1024, 4), (128, 5)):
        print(f"[noalloc] KV E8@2 append {rows}x1024", flush=True)
        x = bf16_rows(rows, 1024, seed, 1.0)
        hq.hq_encode(plan, x, ref, append=total > 0)
        hq.hq_encode_noalloc(plan, x, got, append=total > 0)
        total += rows
        torch.cuda.synchronize()
        same_stream(ref, got, total)


def test_noalloc_largest_call_and_limit(hq):
    """At 2^20 columns (2048 sub-streams per row) 511 rows need 65408
    workgroups, inside the 1 MiB scratch (65528); 513 rows need more and are
    rejected with HQ_ERR_CAPACITY, the stream untouched."""
    cols = 1 << 20
    plan = hq.hq_plan(128, hq.HQ_E8, 4.0, 9, -1, cols)
    assert hq.lib().hq_scan_bytes(plan.handle, 511) <= 1 << 20 < hq.lib().hq_scan_bytes(plan.handle, 513)
    print("[noalloc] E8@4 511x2^20", flush=True)
    x = bf16_rows(513, cols, 6)
    ref = hq.EncodedStream(plan, 511)
    got = hq.EncodedStream(plan, 513)
    hq.hq_encode(plan, x[:511], ref)
    hq.hq_encode_noalloc(plan, x[:511], got)
    torch.cuda.synchronize()
    same_stream(ref, got, 511)
    del ref
    with pytest.raises(hq.HQError) as e:
        hq.hq_encode_noalloc(plan, x, got)
    assert e.value.status == -3
    assert got.rows == 511
