"""Library workspaces under concurrency and stream capture.

The split-tile partials, the expanded block-32 scales and the amax partial
maxima live in library workspaces, one per (device, stream).  Two streams
running the same sequence of calls concurrently must each get the results
of a serial run on one stream, and a sequence captured into a graph on a
stream whose workspaces already exist must reproduce the eager results on
every replay (with eager work on the outputs between replays).  All kernels
here are deterministic, so the bar is bitwise equality with the serial /
eager run; the serial results themselves are checked against the oracle by
the other GPU tests."""

import ctypes

import pytest
import torch

import paper_2609_02846_amd as ue
import synthetic
from tests.gpu_util import say, to_dev

pytestmark = pytest.mark.gpu

# 16 x 17 = 272 tiles of 256 x 256: more than the 256 CUs and a partial last
# wave of 16 tiles, so the fprop runs split tail tiles through the partials
# workspace; K % 512 == 0 keeps the persistent kernel.
T, K, N = 4096, 1024, 4352


def _inputs(seed):
    x = to_dev(synthetic.activation(seed, T, K, 1e-3, 50.0))
    w = to_dev(synthetic.weight(seed, N, K))
    return x, w


def _sequence(x, w, seed, out):
    """amax, SR and RN quantizers, a split-tile GEMM, a block-32 GEMM and a
    running amax, all on the current stream, into the tensors of ``out``."""
    ax, aw = out["ax"], out["aw"]
    ue.amax_accumulate(x, ax, clear=True)
    ue.amax_accumulate(w, aw, clear=True)
    xr = ue.quantize_1d(x, 1, ax, 448.0, "sr", seed, 1, payload=out["xp"], scales=out["xs"], dec_out=out["xd"])
    wq = ue.quantize_2d(w, aw, payload=out["wp"], scales=out["ws"], payload_t=out["wpt"], scales_t=out["wst"],
                        dec_out=out["wd"])
    ue.gemm("nt", T, N, K, *xr, wq[0], wq[1], wq[3], out=out["y"])
    x32 = ue.quantize_1d(x, 1, ax, payload=out["xp32"], scales=out["xs32"], dec_out=out["xd32"], block=32)
    w32 = ue.quantize_2d(w, aw, transposed=False, payload=out["wp32"], scales=out["ws32"], dec_out=out["wd32"],
                         tile=32)
    ue.gemm("nt", T, N, K, *x32, w32[0], w32[1], w32[3], out=out["y32"], out_dtype=torch.bfloat16, block=32)
    ue.amax_accumulate(w, out["arun"], clear=False)


def _buffers():
    u8 = lambda *s: torch.empty(s, dtype=torch.uint8, device="cuda")
    f32 = lambda *s: torch.empty(s, dtype=torch.float32, device="cuda")
    return {"ax": f32(1), "aw": f32(1), "arun": torch.full((1,), 7.0, device="cuda"),
            "xp": u8(T, K // 2), "xs": u8(T, K // 16), "xd": f32(1),
            "wp": u8(N, K // 2), "ws": u8(N // 16, K // 16), "wpt": u8(K, N // 2), "wst": u8(K // 16, N // 16),
            "wd": f32(1), "y": f32(T, N),
            "xp32": u8(T, K // 2), "xs32": u8(T, K // 32), "xd32": f32(1),
            "wp32": u8(N, K // 2), "ws32": u8(N // 32, K // 32), "wd32": f32(1),
            "y32": torch.empty(T, N, dtype=torch.bfloat16, device="cuda")}


def _reset(buf):
    for t in buf.values():
        t.zero_()
    buf["arun"].fill_(7.0)


def _same(a, b, what):
    for k in a:
        assert torch.equal(a[k], b[k]), (what, k)


def test_two_streams_concurrently_equal_serial():
    say("two streams: serial reference")
    ins = [_inputs(1), _inputs(2)]
    ref = [_buffers(), _buffers()]
    for i in range(2):
        _sequence(*ins[i], 100 + i, ref[i])
    torch.cuda.synchronize()
    say("two streams: concurrent")
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    got = [_buffers(), _buffers()]
    for rep in range(3):
        for i in range(2):
            with torch.cuda.stream(streams[i]):
                _sequence(*ins[i], 100 + i, got[i])
        torch.cuda.synchronize()
        for i in range(2):
            _same(got[i], ref[i], f"stream {i} repetition {rep}")
            _reset(got[i])
        torch.cuda.synchronize()


def test_graph_capture_replays_equal_eager():
    """Capture after an eager warm-up on the capturing stream (the
    workspaces exist, so nothing is allocated during capture)."""
    x, w = _inputs(3)
    s = torch.cuda.Stream()
    eager = _buffers()
    say("graph: eager run on the capture stream")
    with torch.cuda.stream(s):
        _sequence(x, w, 7, eager)
    torch.cuda.synchronize()
    cap = _buffers()
    g = torch.cuda.CUDAGraph()
    say("graph: capture")
    with torch.cuda.graph(g, stream=s):
        _sequence(x, w, 7, cap)
    torch.cuda.synchronize()
    for rep in range(3):
        say("graph: replay", rep)
        _reset(cap)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        _same(cap, eager, f"replay {rep}")
        # eager work of the program between replays
        _reset(eager)
        _sequence(x, w, 7, eager)
        torch.cuda.synchronize()


_KEPT_STREAMS = []


class _FreshStream:
    """A new HIP stream (default priority) that no earlier call has used, so
    the library holds no workspace for it yet.  torch's own streams come from
    a pool and are reused, and a destroyed stream's handle value can come
    back from hipStreamCreate (the library would then rightly see the old
    stream's workspaces), so these streams are kept until the process
    ends."""

    def __enter__(self):
        hip = ctypes.CDLL("libamdhip64.so")
        ptr = ctypes.c_void_p()
        assert hip.hipStreamCreate(ctypes.byref(ptr)) == 0
        assert ptr.value not in _KEPT_STREAMS
        _KEPT_STREAMS.append(ptr.value)
        return torch.cuda.ExternalStream(ptr.value)

    def __exit__(self, *exc):
        torch.cuda.synchronize()
        return False


def _split_gemm_operands(seed, k):
    x = to_dev(synthetic.activation(seed, T, k, 1e-3, 50.0))
    w = to_dev(synthetic.weight(seed, N, k))
    ax, aw = torch.empty(1, device="cuda"), torch.empty(1, device="cuda")
    ue.amax_accumulate(x, ax, clear=True)
    ue.amax_accumulate(w, aw, clear=True)
    xr = ue.quantize_1d(x, 1, ax)
    wq = ue.quantize_2d(w, aw, transposed=False)
    return xr, wq


def test_workspace_growth_after_capture_keeps_graph_valid():
    """A graph captured on a stream uses the split-tile workspace that the
    stream held at capture time.  A later, larger split GEMM on that stream
    replaces the workspace; the old buffer stays allocated, so every replay
    of the graph still equals the eager result."""
    with _FreshStream() as s:
        _growth_after_capture(s)


def _growth_after_capture(s):
    with torch.cuda.stream(s):
        small = _split_gemm_operands(4, 1024)       # 272 tiles, 16 split in 2 parts: 8 MiB of partials
        big = _split_gemm_operands(5, 4096)         # 16 split in 8 parts: 32 MiB
        say("growth: eager run of the small split GEMM")
        y_eager = ue.gemm("nt", T, N, 1024, *small[0], small[1][0], small[1][1], small[1][3])
    torch.cuda.synchronize()
    y_cap = torch.zeros_like(y_eager)
    g = torch.cuda.CUDAGraph()
    say("growth: capture the small split GEMM")
    with torch.cuda.graph(g, stream=s):
        ue.gemm("nt", T, N, 1024, *small[0], small[1][0], small[1][1], small[1][3], out=y_cap)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        say("growth: larger split GEMM on the capture stream (new workspace)")
        y_big = ue.gemm("nt", T, N, 4096, *big[0], big[1][0], big[1][1], big[1][3])
        y_big2 = ue.gemm("nt", T, N, 4096, *big[0], big[1][0], big[1][1], big[1][3])
    torch.cuda.synchronize()
    assert torch.equal(y_big, y_big2)
    for rep in range(3):
        say("growth: replay", rep)
        y_cap.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y_cap, y_eager), rep
        with torch.cuda.stream(s):
            y_big3 = ue.gemm("nt", T, N, 4096, *big[0], big[1][0], big[1][1], big[1][3])
        torch.cuda.synchronize()
        assert torch.equal(y_big3, y_big), rep


def test_call_needing_a_workspace_during_capture_is_refused():
    """On a stream that has no split workspace yet, a split GEMM issued
    during capture cannot allocate one: the call fails on the host with
    UE5M3_EHIP and enqueues nothing, and the capture itself stays usable."""
    with _FreshStream() as s:
        _refused_during_capture(s)


def _refused_during_capture(s):
    with torch.cuda.stream(s):
        xr, wq = _split_gemm_operands(6, 1024)
    torch.cuda.synchronize()
    y = torch.zeros(T, N, device="cuda")
    g = torch.cuda.CUDAGraph()
    say("capture: split GEMM on a fresh stream")
    with torch.cuda.graph(g, stream=s):
        with pytest.raises(ue.UE5M3Error) as err:
            ue.gemm("nt", T, N, 1024, *xr, wq[0], wq[1], wq[3], out=y)
        y.add_(1.0)
    assert err.value.status == ue.UE5M3_EHIP
    torch.cuda.synchronize()
    g.replay()
    torch.cuda.synchronize()
    assert torch.all(y == 1.0)
