"""GPU parity of the streaming kernel (hd_infer_stream): a queue of small
batches in one persistent launch, every batch's labels and scores against the
oracle; integer inputs bit-exact; ties; the queue counter and its stop bit."""
import time

import numpy as np
import pytest

import hd_inputs
import oracle
from gpu_util import announce, check_against_oracle, dev, torch_or_skip

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def hd():
    torch_or_skip()
    import paper_2506_09282_amd as hd
    hd.lib()
    return hd


def batches(nbatch, N, F, D, K, dist="uniform_pm1", seed=0):
    X, B, C = hd_inputs.make_inputs(nbatch * N, F, D, K, dist, seed=seed)
    return X.reshape(nbatch, N, F), B, C


def run_stream(hd, X3, B, C, **kw):
    torch = torch_or_skip()
    model = hd.pack_model(dev(B, "f32"), dev(C, "f32"))
    Xd = torch.from_numpy(np.ascontiguousarray(X3)).cuda()
    y, S = hd.infer_stream(Xd, model, return_scores=True, **kw)
    torch.cuda.synchronize()
    return y.cpu().numpy(), S.cpu().numpy().astype(np.float64)


# (nbatch, N, F, D, K): the activity shape at N = 32, 16 and 1 (4-byte X
# pieces: N*F odd), ragged shapes with fewer than 16 samples, many classes,
# and D giving one, two and three blocks per workgroup
STREAM = [(24, 32, 561, 10240, 6), (12, 16, 561, 10240, 6), (40, 1, 561, 10240, 6),
          (9, 7, 300, 3000, 16), (5, 32, 100, 777, 3), (6, 20, 36, 11904, 10),
          (3, 3, 4, 64, 2)]


@pytest.mark.parametrize("nbatch,N,F,D,K", STREAM)
def test_stream_matches_oracle(hd, nbatch, N, F, D, K):
    torch = torch_or_skip()
    assert hd.stream_workspace_bytes(nbatch, N, F, D, K, torch.float32) > 0
    announce(f"stream nbatch={nbatch} N={N} F={F} D={D} K={K}")
    X3, B, C = batches(nbatch, N, F, D, K, seed=nbatch + N)
    y, S = run_stream(hd, X3, B, C)
    X = X3.reshape(nbatch * N, F)
    rep, _ = check_against_oracle(X, B, C, y.reshape(-1), S.reshape(-1, K))
    assert rep["ok"], rep


def test_stream_integer_bit_exact_and_ties(hd):
    announce("stream integer inputs")
    nbatch, N, F, D, K = 10, 32, 561, 10240, 6
    X, B, C = hd_inputs.make_integer_inputs(nbatch * N, F, D, K, seed=4)
    y, S = run_stream(hd, X.reshape(nbatch, N, F), B, C)
    ref = oracle.infer(X, B, C)
    assert np.array_equal(S.reshape(-1, K), ref["S"])
    assert np.array_equal(y.reshape(-1), ref["y"])
    announce("stream ties")
    X, B, C = hd_inputs.make_integer_inputs(6 * 17, 40, 512, 4, seed=3, x_range=1, b_range=1)
    C = np.vstack([C, C[1:2], C[0:1]])
    y, S = run_stream(hd, X.reshape(6, 17, 40), B, C)
    ref = oracle.infer(X, B, C, want_va=True)
    assert (ref["V"] == 0).any()
    assert np.array_equal(S.reshape(-1, 6), ref["S"]) and np.array_equal(y.reshape(-1), ref["y"])


def test_stream_matches_single_batch_calls(hd):
    """Each batch of the stream against hd_infer_packed on that batch alone."""
    torch = torch_or_skip()
    announce("stream vs single-batch calls")
    nbatch, N, F, D, K = 8, 32, 561, 10240, 6
    X3, B, C = batches(nbatch, N, F, D, K, seed=7)
    y, S = run_stream(hd, X3, B, C)
    model = hd.pack_model(dev(B, "f32"), dev(C, "f32"))
    from tolerance import score_scale
    for b in range(nbatch):
        y1, S1 = hd.infer_packed(dev(X3[b], "f32"), model, return_scores=True)
        torch.cuda.synchronize()
        assert np.array_equal(y[b], y1.cpu().numpy())
        assert np.all(np.abs(S[b] - S1.cpu().numpy()) <= 1e-4 * score_scale(C)[None, :])


class _PinnedCounter:
    """A 32-bit counter in coherent pinned host memory (hipHostMalloc), which
    the kernel reads with system-scope loads while the host writes it."""

    def __init__(self):
        import ctypes
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipHostMalloc.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_size_t,
                                           ctypes.c_uint]
        self.hip.hipHostFree.argtypes = [ctypes.c_void_p]
        self.ptr = ctypes.c_void_p()
        rc = self.hip.hipHostMalloc(ctypes.byref(self.ptr), 4, 0x40000000)  # coherent
        assert rc == 0 and self.ptr.value, rc
        self.cell = ctypes.c_uint32.from_address(self.ptr.value)
        self.cell.value = 0

    def data_ptr(self):
        return self.ptr.value

    def set(self, v):
        self.cell.value = v

    def free(self):
        self.hip.hipHostFree(self.ptr)


def test_stream_queue_counter_and_stop(hd):
    """Batches published one by one through a counter in pinned host memory
    while the launch runs; then the stop bit ends the stream early."""
    torch = torch_or_skip()
    nbatch, N, F, D, K = 12, 32, 561, 10240, 6
    announce("stream queue: batches published while the kernel runs")
    X3, B, C = batches(nbatch, N, F, D, K, seed=9)
    model = hd.pack_model(dev(B, "f32"), dev(C, "f32"))
    Xd = torch.from_numpy(X3).cuda()
    ready = _PinnedCounter()
    done = torch.zeros(1, dtype=torch.int32, device="cuda")
    labels = torch.full((nbatch, N), -1, dtype=torch.int32, device="cuda")
    scores = torch.zeros((nbatch, N, K), dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        hd.infer_stream(Xd, model, ready=ready, done=done, out=(labels, scores))
    for b in range(nbatch):
        time.sleep(0.002)
        ready.set(b + 1)
    s.synchronize()
    assert int(done.item()) == nbatch
    X = X3.reshape(-1, F)
    rep, _ = check_against_oracle(X, B, C, labels.cpu().numpy().reshape(-1),
                                  scores.cpu().numpy().astype(np.float64).reshape(-1, K))
    assert rep["ok"], rep

    announce("stream queue: stop after 5 batches")
    ready.set(0)
    done.zero_()
    labels.fill_(-1)
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        hd.infer_stream(Xd, model, ready=ready, done=done, out=(labels, scores))
    ready.set(5)
    time.sleep(0.01)
    ready.set(5 | (1 << 31))
    s.synchronize()
    ready.free()
    assert int(done.item()) == 5
    y = labels.cpu().numpy()
    ref = oracle.infer(X[: 5 * N], B, C)
    assert np.array_equal(y[:5].reshape(-1), ref["y"]) or \
        check_against_oracle(X[: 5 * N], B, C, y[:5].reshape(-1),
                             scores.cpu().numpy().astype(np.float64)[:5].reshape(-1, K))[0]["ok"]
    assert (y[5:] == -1).all()


def test_stream_unsupported_shapes_rejected(hd):
    torch = torch_or_skip()
    # N above 32, K above 16, F above 576, bf16: not served by the stream kernel
    for args in [(4, 33, 561, 10240, 6), (4, 8, 561, 10240, 17), (4, 8, 600, 1024, 6)]:
        assert hd.stream_workspace_bytes(*args, torch.float32) == 0
    assert hd.stream_workspace_bytes(4, 8, 561, 1024, 6, torch.bfloat16) == 0
