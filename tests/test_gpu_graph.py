"""ws_gemm_run under HIP graph capture and on concurrent streams.

A run is one kernel launch on the caller's stream (no memset, no
allocation), so it can be captured: the captured launch is replayed several
times, with eager launches and synchronisations of the program in between,
and every replay must equal the eager result bit for bit.  Two handles on two
streams must not disturb each other."""
import pytest
import torch

from paper_2506_11209_amd import inputs
from tests.gpu_helpers import log

w = pytest.importorskip("paper_2506_11209_amd.wsgemm")

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("shape,tile,stages,np_,nc,epi", [
    ((512, 512, 512), (128, 128, 32), 3, 4, 4, None),                # plain kernel
    ((300, 264, 200), (256, 128, 64), 3, 4, 4, (0.5, 1.0, "bf16")),  # general variant, reads C
    ((256, 256, 0), (128, 128, 32), 3, 4, 4, (1.0, 2.0, "f32")),     # K = 0: the scale kernel
    ((1024, 1024, 448), (256, 128, 64), 3, 4, 4, None),             # deep-prefetch consumer
    ((1024, 512, 512), (128, 64, 64), 4, 8, 4, None),               # the same, 2:1
], ids=["plain", "general", "k0", "deep", "deep-2to1"])
def test_captured_run_replays_equal_eager(shape, tile, stages, np_, nc, epi):
    M, N, K = shape
    log("case graph %s %s" % (shape, epi))
    out = epi[2] if epi else "f32"
    dt = {"f32": torch.float32, "bf16": torch.bfloat16}[out]
    A, B = inputs.make_operands(M, N, K, "bf16", "int4", 61)
    C0 = inputs.make_output(M, N, out, "int4", 62).cuda()
    Ad, Bd = A.cuda(), B.cuda()
    g = w.WsGemm(M, N, K, tile, stages, np_, nc, "bf16")
    try:
        if epi:
            g.set_epilogue(*epi)
        eager = C0.clone()
        g(Ad, Bd, eager)
        torch.cuda.synchronize()
        assert g.sync_status() == w.WS_OK

        C = C0.clone()
        side = torch.cuda.Stream()
        graph = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(graph, stream=side):
            g.run_ptrs(Ad.data_ptr(), Bd.data_ptr(), C.data_ptr(), side.cuda_stream)
        for replay in range(4):
            C.copy_(C0)                   # eager work between replays
            scratch = C0.clone()
            g(Ad, Bd, scratch)            # an eager launch of the same handle
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            assert g.sync_status() == w.WS_OK
            assert torch.equal(C, eager), "replay %d differs from the eager run" % replay
            assert torch.equal(scratch, eager)
        del graph
    finally:
        g.close()


def test_two_handles_on_two_streams():
    log("case two streams")
    A1, B1 = inputs.make_operands(1024, 1024, 512, "bf16", "int4", 71)
    A2, B2 = inputs.make_operands(768, 512, 1024, "f16", "int4", 72)
    g1 = w.WsGemm(1024, 1024, 512, (256, 128, 64), 3, 4, 4, "bf16")
    g2 = w.WsGemm(768, 512, 1024, (128, 128, 32), 3, 8, 4, "f16")
    try:
        A1d, B1d, A2d, B2d = A1.cuda(), B1.cuda(), A2.cuda(), B2.cuda()
        ref1, ref2 = g1(A1d, B1d), g2(A2d, B2d)
        torch.cuda.synchronize()
        s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
        outs = []
        for _ in range(3):
            C1 = torch.empty_like(ref1)
            C2 = torch.empty_like(ref2)
            g1(A1d, B1d, C1, stream=s1)
            g2(A2d, B2d, C2, stream=s2)
            outs.append((C1, C2))
        torch.cuda.synchronize()
        assert g1.sync_status(s1) == w.WS_OK and g2.sync_status(s2) == w.WS_OK
        for C1, C2 in outs:
            assert torch.equal(C1, ref1) and torch.equal(C2, ref2)
    finally:
        g1.close()
        g2.close()
