"""GPU parity of dispatch through bounded destination rings, through the C ABI: the windows
equal the plain dispatch (oracle and xs_dispatch, bit for bit) for ring sizes from one slot
up, with and without per-destination dedup, in device and host-coherent ring memory; the
entry counts equal the oracle's; capacity overflow and argument errors are reported."""
import ctypes as C
import dataclasses

import numpy as np
import pytest
import torch

import synth
from oracle import ep as oep
from oracle import ring as oring
from gpu_helpers import dev_bits, host_bits, require_gpu, xs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()
    torch.cuda.set_device(0)


def _stream():
    return torch.cuda.current_stream().cuda_stream


class Rings:
    """W rings of S slots in device memory, or in host-coherent memory."""

    def __init__(self, T, W, S, H, k, host=False):
        X = xs()
        nb = C.c_int64()
        X.check(X.xs_ring_slot_bytes(H, k, C.byref(nb)))
        self.slot_bytes = nb.value
        self.host = None
        if host:
            from paper_2607_23264_amd.layer import HostCoherent
            self.host = HostCoherent(W * S * self.slot_bytes)
            base = self.host.ptr
            self.arr = X.windows([X.window((base + d * S * self.slot_bytes, S, self.slot_bytes)) for d in range(W)])
        else:
            self.mem = torch.zeros((W, S, self.slot_bytes), dtype=torch.uint8, device="cuda")
            self.arr = X.windows([X.window((self.mem[d].data_ptr(), S, self.slot_bytes)) for d in range(W)])
        X.check(X.xs_dispatch_ring_workspace_bytes(T, k, W, S, C.byref(nb)))
        self.ws = torch.zeros((nb.value,), dtype=torch.uint8, device="cuda")

    def free(self):
        if self.host is not None:
            torch.cuda.synchronize()
            self.host.free()


def _setup(T, H, E, k, W, seed, cap=None):
    g = np.random.default_rng(seed)
    idx = np.argsort(g.random((T, E)), axis=1)[:, :k].astype(np.int32)
    lay = oep.dispatch_layout(idx[None], E, W)
    cap = cap if cap is not None else T * k
    x = synth.normal_bf16(seed, 30, (T, H))
    return idx, lay["slot_row"][0], cap, x


def _ring_dispatch(x, idx, sr, E, W, cap, S, dedup, host=False, max_producers=0, timeout_us=0):
    X = xs()
    T, H = x.shape
    k = idx.shape[1]
    win = torch.full((W, cap, H), -1, dtype=torch.int16, device="cuda")
    wins = X.windows([X.window(win[d]) for d in range(W)])
    rings = Rings(T, W, S, H, k, host)
    st = torch.zeros((1,), dtype=torch.int32, device="cuda")
    stats = torch.full((2 * W,), -1, dtype=torch.int32, device="cuda")
    dx, di, ds = dev_bits(x), torch.from_numpy(idx).cuda(), torch.from_numpy(np.ascontiguousarray(sr)).cuda()
    X.check(X.xs_dispatch_ring(dx.data_ptr(), T, H, di.data_ptr(), ds.data_ptr(), k, E, wins, W, rings.arr, dedup,
                               max_producers, timeout_us, rings.ws.data_ptr(), rings.ws.numel(), stats.data_ptr(),
                               st.data_ptr(), _stream()))
    torch.cuda.synchronize()
    rings.free()
    return host_bits(win), int(st.item()), stats.cpu().numpy()


@pytest.mark.parametrize("S", [1, 2, 5, 64, 4096])
@pytest.mark.parametrize("dedup", [0, 1])
def test_ring_windows_equal_plain_dispatch(S, dedup):
    T, H, E, k, W = 301, 264, 16, 4, 4
    idx, sr, cap, x = _setup(T, H, E, k, W, S + 10 * dedup)
    got, st, stats = _ring_dispatch(x, idx, sr, E, W, cap, S, dedup, max_producers=16)
    assert st == 0
    want, _ = oep.dispatch(x[None], idx[None], sr[None], E, W, cap)
    assert np.array_equal(got, want)
    ent = oring.ring_entries(idx, sr, E, W, bool(dedup))
    assert stats[:W].tolist() == [len(e) for e in ent]
    assert all(0 <= s <= n for s, n in zip(stats[W:], stats[:W]))


@pytest.mark.parametrize("dedup", [0, 1])
def test_ring_host_coherent_memory(dedup):
    T, H, E, k, W = 200, 512, 16, 3, 4
    idx, sr, cap, x = _setup(T, H, E, k, W, 7)
    got, st, _ = _ring_dispatch(x, idx, sr, E, W, cap, 3, dedup, host=True)
    assert st == 0
    want, _ = oep.dispatch(x[None], idx[None], sr[None], E, W, cap)
    assert np.array_equal(got, want)


def test_ring_full_share_equals_oracle_and_xs_dispatch():
    # one source of the DeepSeek-V3-like share: 4096 tokens, H = 7168, top-8 of 256, 8 windows
    X = xs()
    cfg = synth.EP_DSV3_SHARE
    lg = synth.ep_logits(cfg, 0)[0]
    idx, _ = oep.route_topk_softmax(lg, cfg.k)
    lay = oep.dispatch_layout(idx[None], cfg.E, cfg.W)
    sr = lay["slot_row"][0]
    x = synth.ep_x(cfg, 0)[0]
    cap = int(lay["dest_counts"].max())
    plain = torch.full((cfg.W, cap, cfg.H), -1, dtype=torch.int16, device="cuda")
    wins = X.windows([X.window(plain[d]) for d in range(cfg.W)])
    st = torch.zeros((1,), dtype=torch.int32, device="cuda")
    dx, di, ds = dev_bits(x), torch.from_numpy(idx).cuda(), torch.from_numpy(np.ascontiguousarray(sr)).cuda()
    X.check(X.xs_dispatch(dx.data_ptr(), cfg.T, cfg.H, di.data_ptr(), ds.data_ptr(), cfg.k, cfg.E, wins, cfg.W,
                          st.data_ptr(), _stream()))
    torch.cuda.synchronize()
    want = host_bits(plain)
    # the plain dispatch against the oracle's definition, every row of every window
    ref, _ = oep.dispatch(x[None], idx[None], sr[None], cfg.E, cfg.W, cap)
    assert np.array_equal(want, ref)
    for S, dedup in ((16, 1), (16, 0), (1, 1)):
        got, s2, stats = _ring_dispatch(x, idx, sr, cfg.E, cfg.W, cap, S, dedup)
        assert s2 == 0 and int(st.item()) == 0
        assert np.array_equal(got, want), (S, dedup)
        ent = oring.ring_entries(idx, sr, cfg.E, cfg.W, bool(dedup))
        assert stats[:cfg.W].tolist() == [len(e) for e in ent]


def test_ring_capacity_overflow():
    X = xs()
    T, H, E, k, W = 64, 64, 4, 2, 2
    idx, sr, _, x = _setup(T, H, E, k, W, 9)
    got, st, _ = _ring_dispatch(x, idx, sr, E, W, 20, 2, 1)
    assert st == X.XS_ECAPACITY
    want, _ = oep.dispatch(x[None], idx[None], sr[None], E, W, 20)
    assert np.array_equal(got, want)


def test_ring_time_out_path_exits_and_recovers():
    # a 1 us bound on every wait: the run either completes or gives up with XS_ETIMEOUT, and
    # either way the kernel exits; a following call with the default bound is whole
    X = xs()
    T, H, E, k, W = 400, 1024, 16, 4, 4
    idx, sr, cap, x = _setup(T, H, E, k, W, 11)
    _, st, _ = _ring_dispatch(x, idx, sr, E, W, cap, 1, 1, timeout_us=1)
    assert st in (0, X.XS_ETIMEOUT)
    got, st, _ = _ring_dispatch(x, idx, sr, E, W, cap, 1, 1)
    assert st == 0
    want, _ = oep.dispatch(x[None], idx[None], sr[None], E, W, cap)
    assert np.array_equal(got, want)


def test_ring_bad_arguments():
    X = xs()
    T, H, E, k, W = 8, 64, 4, 2, 2
    idx, sr, cap, x = _setup(T, H, E, k, W, 1)
    win = torch.zeros((W, cap, H), dtype=torch.int16, device="cuda")
    wins = X.windows([X.window(win[d]) for d in range(W)])
    r = Rings(T, W, 4, H, k)
    st = torch.zeros((1,), dtype=torch.int32, device="cuda")
    dx, di, ds = dev_bits(x), torch.from_numpy(idx).cuda(), torch.from_numpy(np.ascontiguousarray(sr)).cuda()

    def call(rings=r.arr, ws=r.ws.numel(), kk=k, dedup=1, HH=H):
        return X.xs_dispatch_ring(dx.data_ptr(), T, HH, di.data_ptr(), ds.data_ptr(), kk, E, wins, W, rings, dedup,
                                  0, 0, r.ws.data_ptr(), ws, None, st.data_ptr(), _stream())

    assert call(ws=r.ws.numel() - 4) == X.XS_EWORKSPACE
    assert call(dedup=2) == X.XS_EINVAL
    assert call(kk=33) == X.XS_EINVAL
    assert call(HH=60) == X.XS_EUNSUPPORTED
    small = X.windows([X.window((r.arr[d].base, 4, r.slot_bytes - 16)) for d in range(W)])
    assert call(rings=small) == X.XS_EINVAL
    mixed = X.windows([X.window((r.arr[d].base, 4 if d == 0 else 3, r.slot_bytes)) for d in range(W)])
    assert call(rings=mixed) == X.XS_EINVAL
    torch.cuda.synchronize()
    assert int(st.item()) == 0
