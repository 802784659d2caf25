"""si_selective_ffn, si_selective_ffn_resnorm and si_dynamic_set captured in a HIP graph (as
the benchmark times them): each replay, with other eager work on the stream in between, must
give the eager call's result bit for bit (every reduction has a fixed order). No entry point on
these paths records a memset or an allocation, so a replay repeats exactly the eager kernels."""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_18081_amd as si
from tests.gpu_util import dev_tensor, host_array, max_rel_l2, say
from workloads import csr_from_sets

pytestmark = pytest.mark.gpu


def _problem(seed, N, d, L, B, wdtype="bf16"):
    rng = np.random.default_rng(seed)

    def draw(*shape, scale=0.02):
        a = (rng.standard_normal(shape) * scale).astype(np.float32)
        return (a.view(np.uint32) >> 16).astype(np.uint16) if wdtype == "bf16" else a

    wg, wu, wd = draw(N, d), draw(N, d), draw(d, N)
    loaded = rng.permutation(N)[:L].astype(np.int32)
    ref = oracle.compact(wg, wu, wd, loaded)
    gpu = si.compact_ffn(dev_tensor(wg), dev_tensor(wu), dev_tensor(wd), torch.from_numpy(loaded))
    sets = [rng.permutation(L)[:int(rng.integers(0, L + 1)) if b % 3 else 40].astype(np.int32)
            for b in range(B)]
    x = draw(B, d, scale=1.0)
    return rng, ref, gpu, sets, x


@pytest.mark.parametrize("B,d,L,wdtype,flags", [
    (1, 1000, 530, "bf16", 0),              # per-token gather-GEMV + reducer
    (3, 264, 530, "f32", 0),                # per-token, several tokens
    (16, 264, 613, "bf16", 0),              # union path, row-word kernels
    (2, 264, 613, "bf16", si.FLAG_UNION),   # the same below 5 tokens
    (130, 264, 613, "bf16", 0),             # union path, LDS-tiled GEMMs
])
def test_graph_replay_selective_ffn(B, d, L, wdtype, flags):
    say(f"graph replay B={B} d={d} L={L} {wdtype} flags={flags}")
    rng, ref, gpu, sets, x = _problem(B * 13 + d, L + 170, d, L, B, wdtype)
    off, idx = csr_from_sets(sets)
    xd, offd, idxd = dev_tensor(x), dev_tensor(off), dev_tensor(idx)
    need = si.selective_ffn_workspace(B, idx.size, L, d, si.BF16 if wdtype == "bf16" else si.F32,
                                      si.BF16 if wdtype == "bf16" else si.F32, flags)
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device="cuda:0")
    eager = host_array(si.selective_ffn(xd, offd, idxd, gpu.gate_up_c, gpu.down_c, flags=flags,
                                        workspace=ws))
    want = np.stack([oracle.selective_ffn(x[b], sets[b], ref["gate_up_c"], ref["down_c"])
                     for b in range(B)])
    assert max_rel_l2(eager, want) <= (5e-3 if wdtype == "bf16" else 1e-5)
    y = torch.empty((B, d), dtype=torch.float32, device="cuda:0")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        si.selective_ffn(xd, offd, idxd, gpu.gate_up_c, gpu.down_c, flags=flags, y=y,
                         workspace=ws)
    # other work on the same buffers between replays: an eager call with another input
    x2 = dev_tensor(x[::-1].copy())
    other = torch.empty_like(y)
    for rep in range(3):
        y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(host_array(y), eager), f"replay {rep}"
        si.selective_ffn(x2, offd, idxd, gpu.gate_up_c, gpu.down_c, flags=flags, y=other,
                         workspace=ws)
        torch.cuda.synchronize()


def test_graph_replay_resnorm():
    say("graph replay of si_selective_ffn_resnorm (stacked layer)")
    B, d, L = 1, 4104, 530
    rng, ref, gpu, sets, x = _problem(77, L + 170, d, L, B)
    off, idx = csr_from_sets(sets)
    offd, idxd = dev_tensor(off), dev_tensor(idx)
    xp = dev_tensor(x)
    yp = dev_tensor((rng.standard_normal((B, d)) * 0.3).astype(np.float32))
    need = si.selective_ffn_workspace(B, idx.size, L, d)
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device="cuda:0")
    xo_e, y_e = si.selective_ffn_resnorm(xp, yp, offd, idxd, gpu.gate_up_c, gpu.down_c,
                                         workspace=ws)
    xo_e, y_e = host_array(xo_e), host_array(y_e)
    xo = torch.empty_like(xp)
    y = torch.empty((B, d), dtype=torch.float32, device="cuda:0")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        si.selective_ffn_resnorm(xp, yp, offd, idxd, gpu.gate_up_c, gpu.down_c, x_out=xo, y=y,
                                 workspace=ws)
    for rep in range(3):
        xo.zero_()
        y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(host_array(xo), xo_e) and np.array_equal(host_array(y), y_e), rep
        si.selective_ffn(xp, offd, idxd, gpu.gate_up_c, gpu.down_c, workspace=ws)
        torch.cuda.synchronize()


@pytest.mark.parametrize("L", [530, 33000])
def test_graph_replay_dynamic_set(L):
    """si_dynamic_set in a graph: the bitmap path (up to 32768 slots) and the list path past
    it. No step records a memset, so each replay repeats the eager result bit for bit."""
    say(f"graph replay of si_dynamic_set L={L}")
    T, d = 40, 64
    rng, ref, gpu, _, _ = _problem(L, L + 170, d, L, 1)
    xb = (rng.standard_normal((T, d)).astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    x = dev_tensor(xb)
    static = dev_tensor(rng.permutation(L)[:L // 8].astype(np.int32))
    alpha, n_total = L // 5, L // 3
    need = int(si._lib.load().si_dynamic_set_workspace(T, L, alpha, n_total))
    ws = torch.empty(need, dtype=torch.uint8, device="cuda:0")
    out_e, cnt_e = si.dynamic_set(x, gpu.gate_up_c, static, alpha, n_total, workspace=ws)
    out_e, cnt_e = host_array(out_e), host_array(cnt_e)
    out = torch.empty(n_total, dtype=torch.int32, device="cuda:0")
    cnt = torch.empty(L, dtype=torch.int32, device="cuda:0")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        si.dynamic_set(x, gpu.gate_up_c, static, alpha, n_total, workspace=ws, out=out, counts=cnt)
    x2 = dev_tensor(xb[::-1].copy())
    for rep in range(3):
        out.fill_(-7)
        cnt.fill_(-7)
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(host_array(out), out_e), rep
        assert np.array_equal(host_array(cnt), cnt_e), rep
        si.dynamic_set(x2, gpu.gate_up_c, static, alpha, n_total, workspace=ws)
        torch.cuda.synchronize()
