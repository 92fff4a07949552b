"""The codec under HIP graph capture (torch.cuda.CUDAGraph over the caller's
stream): encode and decode launches, the group launches, an encode followed
by appends, and the no-allocation encode are captured once and replayed
several times, with eager work and synchronizations between the replays;
every replay's stream words, offsets, k bytes, norms and decoded values
equal the eager run's.  The look-back's launch epoch lives in device memory
and advances on every replay, so the statuses of one replay never satisfy
the next one's waits."""
import pytest
import torch

from oracle import oracle as O
from tests import parity as PT
from tests.test_gpu_tiles import gauss

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def hq():
    from paper_2606_23406_amd import hq as H
    H.lib()
    assert torch.cuda.is_available()
    return H


def snapshot(s, rows):
    spr = s.plan.info.subs_per_row
    end = int(s.offsets[rows * spr].item())
    return (s.payload[:end].clone(), s.offsets[: rows * spr + 1].clone(),
            s.kparam[: rows * spr].clone(), s.norms.clone())


def test_encode_decode_replays(hq):
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=3)
    x = gauss(96, 4096, 11).cuda()
    plan = PT.gpu_plan(hq, P, snr, 4096)
    s = hq.EncodedStream(plan, 96)
    y = torch.empty_like(x)
    print("[graph] encode + decode 96x4096", flush=True)

    def run():
        hq.hq_encode(plan, x, s)
        hq.hq_decode(plan, s, out=y)

    def scribble():
        s.payload.fill_(0xAB)
        y.fill_(0.0)

    check = [lambda: snapshot(s, 96), lambda: y.clone()]
    run()
    torch.cuda.synchronize()
    ref = [c() for c in check]
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side), torch.cuda.graph(g):
        run()
    torch.cuda.current_stream().wait_stream(side)
    for r in range(4):
        scribble()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = [c() for c in check]
        for a, b in zip(ref[0], got[0]):
            assert torch.equal(a, b), f"stream differs on replay {r}"
        assert torch.equal(ref[1], got[1]), f"decode differs on replay {r}"
        assert s.read_stats()["status"] == 0


def test_appends_and_noalloc_replay(hq):
    # a fresh block and three appends (KV plan: signs, dither, fp16 norms),
    # encoded through the no-allocation entry point, then decoded
    snr = 10.0
    P = PT.oracle_params(O.E8, snr, rht_seed=5, rotation=1, rot_seed=6, dither=True, dither_seed=7,
                         norm_fp16=True)
    x = gauss(4 * 256, 1024, 13, scale=1.0).cuda()
    plan = PT.gpu_plan(hq, P, snr, 1024)
    s = hq.EncodedStream(plan, 4 * 256)
    y = torch.empty_like(x)
    print("[graph] noalloc encode + 3 appends + decode, 1024x1024 KV", flush=True)

    def run():
        for b in range(4):
            hq.hq_encode_noalloc(plan, x[b * 256:(b + 1) * 256], s, append=b > 0)
        hq.hq_decode(plan, s, out=y)

    run()
    torch.cuda.synchronize()
    ref = (snapshot(s, 1024), y.clone())
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side), torch.cuda.graph(g):
        run()
    torch.cuda.current_stream().wait_stream(side)
    for r in range(3):
        s.payload.fill_(0)
        s.offsets.fill_(0)
        y.fill_(1.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        snap = snapshot(s, 1024)
        for a, b in zip(ref[0], snap):
            assert torch.equal(a, b), f"stream differs on replay {r}"
        assert torch.equal(ref[1], y), f"decode differs on replay {r}"


def test_group_launch_replays(hq):
    snr = PT.op_snr("E8", 4.0)
    P = PT.oracle_params(O.E8, snr, rht_seed=8)
    plan = PT.gpu_plan(hq, P, snr, 2048)
    xs = [gauss(r, 2048, 20 + r).cuda() for r in (40, 9, 130)]
    ss = [hq.EncodedStream(plan, x.shape[0]) for x in xs]
    ys = [torch.empty_like(x) for x in xs]
    print("[graph] group encode + decode, 3 matrices", flush=True)

    def run():
        hq.hq_encode_group([plan] * 3, xs, ss)
        hq.hq_decode_group([plan] * 3, ss, ys)

    run()
    torch.cuda.synchronize()
    ref = [(snapshot(s, x.shape[0]), y.clone()) for s, x, y in zip(ss, xs, ys)]
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side), torch.cuda.graph(g):
        run()
    torch.cuda.current_stream().wait_stream(side)
    for r in range(3):
        for s, y in zip(ss, ys):
            s.payload.fill_(0x55)
            y.fill_(-1.0)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for (rs, ry), s, x, y in zip(ref, ss, xs, ys):
            for a, b in zip(rs, snapshot(s, x.shape[0])):
                assert torch.equal(a, b), f"stream differs on replay {r}"
            assert torch.equal(ry, y), f"decode differs on replay {r}"
