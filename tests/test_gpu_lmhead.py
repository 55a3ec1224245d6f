"""GPU parity of lmhead_logsoftmax_verify against the fp64 oracle (C ABI)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_36546_amd import inputs, ops
from tests import parity
from tests.workload import to_np

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _run(hidden, W, prop, K, out_rows=None, n_out=None):
    outs = ops.lmhead_logsoftmax_verify(hidden, W, prop, K, out_rows=out_rows, n_out_rows=n_out)
    torch.cuda.synchronize()
    return outs


def _check(hidden, W, prop_np, K):
    dev = hidden.device
    prop = torch.from_numpy(prop_np.astype(np.int32)).to(dev)
    g = _run(hidden, W, prop, K)
    logits = oracle.logits_fp64(to_np(hidden), to_np(W))
    ref = oracle.lmhead_logsoftmax(None, None, prop_np, K, logits=logits)
    c = parity.check_lmhead(g, ref, logits, K)
    _say(f"  rows={c['rows']} excluded(set margin<=1e-3)={c['excluded']}")
    return g, ref, logits


def _rand(M, Hd, V, dtype, seed, std=0.02):
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    h = torch.randn(M, Hd, generator=gen, device="cuda")
    h = (h / h.pow(2).mean(1, keepdim=True).sqrt()).to(dtype)
    W = (torch.randn(V, Hd, generator=gen, device="cuda") * std).to(dtype)
    prop = np.random.default_rng(seed).integers(0, V, size=M)
    return h, W, prop


def test_tiny_fp32_config():
    _say("[lmhead] tiny fp32 M=8 Hd=256 V=1024 K=16")
    h, W, prop = _rand(8, 256, 1024, torch.float32, 1)
    _check(h, W, prop, 16)


@pytest.mark.parametrize("M,Hd,V,K", [(40, 2048, 151936, 16), (300, 256, 5003, 32),
                                      (1, 64, 64, 1), (129, 512, 2048, 4), (33, 128, 100, 32),
                                      (7, 4096, 262144, 16), (3, 4096, 262143, 32),
                                      (100, 256, 151936, 16), (160, 256, 151936, 8),
                                      (700, 256, 50000, 16), (1024, 128, 30000, 8)])
def test_bf16_shapes(M, Hd, V, K):
    """Includes the largest supported shape (V = 262144, Hd = 4096) and a
    ragged last group at that size.  M = 100 and 160 take the 128-row and the
    192-row tiles with 594 vocabulary tiles, so every persistent workgroup
    runs two or three tiles (M = 40, 7 and 3 do so with 64-row tiles).  M =
    700 and 1024 have three and four 256-row tiles (the last one ragged at
    700), 588 and 472 tile numbers, so a workgroup's walk crosses row tiles."""
    _say(f"[lmhead] bf16 M={M} Hd={Hd} V={V} K={K}")
    h, W, prop = _rand(M, Hd, V, torch.bfloat16, M + V)
    _check(h, W, prop, K)


def test_fp32_ragged():
    _say("[lmhead] fp32 M=70 Hd=128 V=3001 K=8")
    h, W, prop = _rand(70, 128, 3001, torch.float32, 7, std=0.3)
    _check(h, W, prop, 8)


def test_uniform_logits_tie_break():
    """W = 0: every logit ties; top-K must be indices 0..K-1, argmax 0,
    logp = -log V, entropy = log V."""
    V, K = 4096, 32
    h = torch.ones(5, 128, device="cuda", dtype=torch.bfloat16)
    W = torch.zeros(V, 128, device="cuda", dtype=torch.bfloat16)
    prop = torch.tensor([0, 31, 32, 4095, 7], dtype=torch.int32, device="cuda")
    g = _run(h, W, prop, K)
    np.testing.assert_array_equal(to_np(g["topk_idx"]), np.tile(np.arange(K), (5, 1)))
    np.testing.assert_array_equal(to_np(g["argmax"]), 0)
    np.testing.assert_allclose(to_np(g["logp_prop"]), -np.log(V), atol=1e-4)
    np.testing.assert_allclose(to_np(g["entropy"]), np.log(V), atol=1e-3)


def test_duplicated_rows_and_clusters():
    """Many exact ties and several top-K members inside one 64-entry group."""
    V, Hd, K = 2048, 64, 16
    gen = torch.Generator(device="cuda")
    gen.manual_seed(3)
    W = torch.randn(V, Hd, generator=gen, device="cuda") * 0.05
    W[100:110] = W[5]            # ten copies of one row in one group
    W[1500] = W[5]
    h = torch.zeros(3, Hd, device="cuda")
    h[:] = W[5] * 20
    h, W = h.to(torch.bfloat16), W.to(torch.bfloat16)
    prop = np.array([109, 1500, 3])
    g, ref, logits = _check(h, W, prop, K)
    top = to_np(g["topk_idx"])[0].tolist()
    assert top[:12] == [5] + list(range(100, 110)) + [1500]


def test_out_rows_scatter():
    h, W, prop = _rand(20, 256, 3000, torch.bfloat16, 9)
    rows = torch.tensor(np.random.default_rng(0).permutation(50)[:20].astype(np.int32), device="cuda")
    p = torch.from_numpy(prop.astype(np.int32)).cuda()
    a = _run(h, W, p, 8)
    b = _run(h, W, p, 8, out_rows=rows, n_out=50)
    r = rows.long()
    for key in ("lse", "logp_prop", "argmax", "topk_idx", "topk_logp", "entropy"):
        assert torch.equal(a[key], b[key][r]), key


def test_full_size_teacher_rows_sampled():
    """The full LM head shape (512 rows, V=151936, Hd=2048) as the benchmark
    launches it; the oracle checks 24 sampled rows."""
    _say("[lmhead] full teacher shape M=512, oracle on 24 rows")
    h, W, prop = _rand(512, 2048, 151936, torch.bfloat16, 512)
    p = torch.from_numpy(prop.astype(np.int32)).cuda()
    g = _run(h, W, p, 16)
    rows = np.random.default_rng(1).choice(512, 24, replace=False)
    rows.sort()
    logits = oracle.logits_fp64(to_np(h[torch.from_numpy(rows).cuda()]), to_np(W))
    ref = oracle.lmhead_logsoftmax(None, None, prop[rows], 16, logits=logits)
    sub = {k: (v[torch.from_numpy(rows).cuda()] if v is not None else None) for k, v in g.items()}
    c = parity.check_lmhead(sub, ref, logits, 16)
    _say(f"  excluded {c['excluded']} of {c['rows']}")


def test_recompute_with_a_long_survivor_list():
    """Ten groups each hold four of the top-32 logits, so the merge recomputes
    all ten (1280 logits); 1470 other records tie at the lower bound theta
    and survive, so the survivors and the recomputed logits together exceed
    the merge's list and it must select from all group records.  Logits are
    exact (one non-zero channel), the ties are broken by index, so the top-K
    list is unique and compared in full."""
    V, Hd, K = 64000, 64, 32
    _say(f"[lmhead] long survivor list with recompute V={V} K={K}")
    W = torch.zeros(V, Hd)
    W[:, 0] = 0.5                                    # every other logit: 0.5
    for grp in range(10):                            # groups 0..9: four members each
        W[grp * 128 + 0, 0] = 4.0
        W[grp * 128 + 1, 0] = 3.0
        W[grp * 128 + 2, 0] = 2.0
        W[grp * 128 + 3, 0] = 1.0 + grp / 16.0       # the fourth members rank by group
    h = torch.zeros(2, Hd)
    h[:, 0] = 1.0
    h, W = h.cuda().to(torch.bfloat16), W.cuda().to(torch.bfloat16)
    prop = np.array([3, 9 * 128 + 3])
    g, ref, logits = _check(h, W, prop, K)
    want = ([grp * 128 for grp in range(10)] + [grp * 128 + 1 for grp in range(10)]
            + [grp * 128 + 2 for grp in range(10)] + [9 * 128 + 3, 8 * 128 + 3])
    for r in range(2):
        assert to_np(g["topk_idx"])[r].tolist() == want
        assert ref["topk_idx"][r].tolist() == want
