"""si_selective_ffn_noalloc (the entry point for callers that cannot allocate) against
si_selective_ffn, through the C ABI.

Both run the same kernels on the same inputs, one with a caller workspace and one with the
library's static device scratch, so the outputs must be bitwise equal. Each case makes two
calls in a row, the second with a smaller input (fewer tokens, a shorter active list), so a
result that leaned on the first call's scratch contents would show. A request whose workspace
exceeds the scratch is refused with SI_ERR_UNSUPPORTED before anything is enqueued.
"""
import numpy as np
import pytest
import torch

import paper_2607_18081_amd as si
from tests.gpu_util import dev_tensor, host_array, say
from workloads import csr_from_sets

pytestmark = pytest.mark.gpu


def _layer(seed, N, d, L):
    rng = np.random.default_rng(seed)
    def draw(*shape, scale=0.02):
        a = (rng.standard_normal(shape) * scale).astype(np.float32)
        return (a.view(np.uint32) >> 16).astype(np.uint16)
    wg, wu, wd = draw(N, d), draw(N, d), draw(d, N)
    loaded = rng.permutation(N)[:L].astype(np.int32)
    gpu = si.compact_ffn(dev_tensor(wg), dev_tensor(wu), dev_tensor(wd), torch.from_numpy(loaded))
    return rng, draw, gpu


def _pair(x, sets, gpu, flags=0):
    off, idx = csr_from_sets(sets)
    xd, od, idd = dev_tensor(x), dev_tensor(off), dev_tensor(idx)
    want = si.selective_ffn(xd, od, idd, gpu.gate_up_c, gpu.down_c, flags=flags)
    y = torch.full((x.shape[0], x.shape[1]), float("nan"), dtype=torch.float32, device="cuda:0")
    got = si.selective_ffn_noalloc(xd, od, idd, gpu.gate_up_c, gpu.down_c, y, flags=flags)
    torch.cuda.synchronize()
    return host_array(got), host_array(want)


@pytest.mark.parametrize("B1,B2,flags", [(1, 1, 0), (16, 6, 0), (4, 2, si.FLAG_UNION),
                                          (160, 130, 0), (160, 130, si.FLAG_EXACT_H),
                                          (3, 1, si.FLAG_PER_TOKEN)])
def test_noalloc_matches_selective_ffn(B1, B2, flags):
    N, d, L = 3000, 2048, 2100
    say(f"noalloc: B={B1} then B={B2}, flags={flags}")
    rng, draw, gpu = _layer(B1 * 7 + B2, N, d, L)
    for B, k in ((B1, 700), (B2, 150)):          # the second call is smaller
        sets = [rng.permutation(L)[:k - 13 * (b % 5)].astype(np.int32) for b in range(B)]
        x = draw(B, d, scale=1.0)
        got, want = _pair(x, sets, gpu, flags)
        assert np.array_equal(got, want), (B, k)
        assert np.all(np.isfinite(got))


def test_noalloc_refuses_oversized_requests():
    """A workspace need past the static scratch is refused; the same call with a workspace of
    its own still runs."""
    say("noalloc: oversized request refused")
    lib = si._lib.load()
    B, d, L = 4096, 4096, 9000
    need = lib.si_selective_ffn_workspace(B, B * 10, L, d, si.BF16, si.BF16, 0)
    assert need > si.api.NOALLOC_SCRATCH_BYTES
    x = torch.zeros((B, d), dtype=torch.bfloat16, device="cuda:0")
    off = torch.zeros(B + 1, dtype=torch.int32, device="cuda:0")
    idx = torch.zeros(1, dtype=torch.int32, device="cuda:0")
    gu = torch.zeros((L, 2, d), dtype=torch.bfloat16, device="cuda:0")
    dn = torch.zeros((L, d), dtype=torch.bfloat16, device="cuda:0")
    y = torch.zeros((B, d), dtype=torch.float32, device="cuda:0")
    with pytest.raises(si.SelectInferError) as e:
        si.selective_ffn_noalloc(x, off, idx, gu, dn, y)
    assert e.value.status == 5


def test_noalloc_7b_decode_shape():
    """The 7B decode shape (d = 4096, 2202 active rows), twice in a row, then 1100 rows."""
    say("noalloc: 7B decode shape")
    rng, draw, gpu = _layer(11, 11008, 4096, 7706)
    for k in (2202, 2202, 1100):
        sets = [rng.permutation(7706)[:k].astype(np.int32)]
        got, want = _pair(draw(1, 4096, scale=1.0), sets, gpu)
        assert np.array_equal(got, want)
