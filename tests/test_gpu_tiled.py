"""The tiled weight layout (lmhead_pack_w, IPDV_W_TILED) on the GPU.

The tiled GEMM loads each 16-row x 32-channel block as one contiguous 1 KB
run but writes the same bytes to LDS as the row-major path, and every other
read of W goes through the same element mapping; so every output must be
bit-identical to the row-major call (which the other GPU tests check against
the oracle).  One shape is also checked against the oracle directly."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36546_amd import ops
from tests import parity
from tests.workload import to_np

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _rand(M, Hd, V, seed, std=0.02):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    h = torch.randn(M, Hd, generator=g, device="cuda")
    h = (h / h.pow(2).mean(1, keepdim=True).sqrt()).to(torch.bfloat16)
    W = (torch.randn(V, Hd, generator=g, device="cuda") * std).to(torch.bfloat16)
    return h, W


@pytest.mark.parametrize("V,Hd", [(1003, 128), (151936, 2048), (16, 64)])
def test_pack_layout(V, Hd):
    _say(f"[tiled] pack V={V} Hd={Hd}")
    _, W = _rand(1, Hd, V, V)
    P = ops.lmhead_pack_w(W)
    torch.cuda.synchronize()
    Vp = -(-V // 16) * 16
    Wpad = torch.zeros(Vp, Hd, dtype=W.dtype, device=W.device)
    Wpad[:V] = W
    ref = Wpad.view(Vp // 16, 16, Hd // 32, 32).permute(0, 2, 1, 3).contiguous().view(-1)
    assert P.data.numel() == ref.numel()
    assert torch.equal(P.data, ref)


def _lm(h, W, prop, K):
    ws = torch.empty(ops.lmhead_workspace_size(h.shape[0], h.shape[1],
                                               W.V if isinstance(W, ops.PackedW) else W.shape[0], K),
                     dtype=torch.uint8, device=h.device)
    outs = ops.lmhead_logsoftmax_verify(h, W, prop, K, workspace=ws)
    return outs, ws


@pytest.mark.parametrize("M,Hd,V,K", [(40, 2048, 151936, 16), (129, 512, 2048, 4),
                                      (7, 4096, 262143, 32), (33, 128, 100, 32), (1, 64, 64, 1),
                                      (512, 2048, 151936, 16)])
def test_lmhead_tiled_equals_row_major(M, Hd, V, K):
    _say(f"[tiled] lmhead M={M} Hd={Hd} V={V} K={K}")
    h, W = _rand(M, Hd, V, M + V)
    P = ops.lmhead_pack_w(W)
    prop = torch.from_numpy(np.random.default_rng(M).integers(0, V, size=M).astype(np.int32)).cuda()
    a, ws_a = _lm(h, W, prop, K)
    b, ws_b = _lm(h, P, prop, K)
    torch.cuda.synchronize()
    for k in a:
        assert torch.equal(a[k], b[k]), k
    # the draws and the gather read W too
    u = torch.from_numpy(((np.arange(M) + 0.5) / M).astype(np.float32)).cuda()
    ta = ops.lmhead_sample(h, W, K, ws_a, u)
    tb = ops.lmhead_sample(h, P, K, ws_b, u)
    idx = torch.from_numpy(np.random.default_rng(1).integers(-2, V + 2, size=(M, 24)).astype(np.int32)).cuda()
    ga = ops.lmhead_logp_gather(h, W, a["lse"], idx)
    gb = ops.lmhead_logp_gather(h, P, b["lse"], idx)
    cu = torch.arange(M + 1, dtype=torch.int32, device="cuda")
    drv = torch.zeros(M, dtype=torch.uint8, device="cuda")
    ev = torch.zeros(M, dtype=torch.int32, device="cuda")
    fa = torch.zeros(M, dtype=torch.uint8, device="cuda")
    fb = torch.zeros(M, dtype=torch.uint8, device="cuda")
    sa = ops.sample_takeover(h, W, K, ws_a, cu, drv, ev, u, V - 1, fa)
    sb = ops.sample_takeover(h, P, K, ws_b, cu, drv, ev, u, V - 1, fb)
    torch.cuda.synchronize()
    assert torch.equal(ta, tb) and torch.equal(ga, gb) and torch.equal(sa, sb) and torch.equal(fa, fb)


def test_tiled_recompute_path_and_oracle():
    """Four equal rows inside one 128-entry group put four of a row's top-K in
    one group, which forces the merge's exact recompute from W; the tiled
    call must agree with the row-major one and with the oracle."""
    _say("[tiled] recompute path V=5003 Hd=256")
    M, Hd, V, K = 16, 256, 5003, 8
    h, W = _rand(M, Hd, V, 77, std=0.05)
    W[260:264] = (h[0] * 0.4).to(W.dtype)            # four equal, large rows in group 2
    P = ops.lmhead_pack_w(W)
    prop = torch.full((M,), 261, dtype=torch.int32, device="cuda")
    a, _ = _lm(h, W, prop, K)
    b, _ = _lm(h, P, prop, K)
    torch.cuda.synchronize()
    for k in a:
        assert torch.equal(a[k], b[k]), k
    logits = oracle.logits_fp64(to_np(h), to_np(W))
    ref = oracle.lmhead_logsoftmax(None, None, np.full(M, 261), K, logits=logits)
    parity.check_lmhead(b, ref, logits, K)
    assert set(to_np(b["topk_idx"])[0][:4].tolist()) == {260, 261, 262, 263}
