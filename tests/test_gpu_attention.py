"""GPU parity of verify_attn_paged (append + causal paged attention) against
the fp64 oracle, called through the C ABI."""
import numpy as np
import pytest
import torch

from paper_2609_36546_amd import inputs, ops
from tests import parity
from tests.workload import to_np

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _case(cfg, seed=0, **kw):
    _say(f"[attn] cfg={cfg.name} B={cfg.B} ctx=[{cfg.ctx_lo},{cfg.ctx_hi}] k={cfg.k_choices} "
         f"ps={cfg.page_size} seed={seed}")
    return inputs.make_batch(cfg, seed=seed, device="cuda", **kw)


def _check_all(batch, mi=0):
    mdl = batch.models[mi]
    seqs = to_np(mdl.seq_ids).astype(np.int64)
    D = mdl.shape.D
    out, kc, vc = parity.run_gpu_attention(mdl, batch, seq_ids=mdl.seq_ids)
    ref, rkc, rvc = parity.oracle_attention(mdl, batch, seqs, D)
    rows = to_np(mdl.rows).astype(np.int64)
    worst = parity.check_attention_rows(out, ref, rows, mdl.q.dtype)
    # the window was appended bit-exactly and nothing else in the pools changed
    np.testing.assert_array_equal(to_np(kc), rkc.astype(np.float32))
    np.testing.assert_array_equal(to_np(vc), rvc.astype(np.float32))
    _say(f"  worst rel err {worst:.2e} over {len(rows)} rows")
    return worst


def test_tiny_fp32_config():
    _check_all(_case(inputs.WORKLOADS["tiny-f32"]))


@pytest.mark.parametrize("name,B,lo,hi,seed", [("student-bf16", 5, 40, 1500, 2),
                                               ("teacher-bf16", 4, 100, 2600, 3),
                                               ("teacher-bf16", 3, 1, 40, 3)])
def test_scaled_bf16_configs(name, B, lo, hi, seed):
    base = inputs.WORKLOADS[name]
    cfg = inputs.scaled(base, B=B, ctx_lo=lo, ctx_hi=hi,
                        models=(inputs.scaled_shape(base.models[0], vocab=512, hidden=64),))
    _check_all(_case(cfg, seed=seed))


def test_long_window_two_row_groups():
    """k = 16 with 8 query heads per KV head: 128 packed rows, two row groups."""
    cfg = inputs.scaled(inputs.WORKLOADS["long-teacher-bf16"], B=2, ctx_lo=3000, ctx_hi=5200, pool_tokens=None,
                        models=(inputs.scaled_shape(inputs.TEACHER, vocab=512, hidden=64),))
    _check_all(_case(cfg, seed=4))


@pytest.mark.parametrize("B,ks,lo,hi,seed", [(12, (0, 1, 8, 16), 0, 300, 7),
                                              (60, (0, 4, 16), 0, 40, 8)])
def test_empty_windows_and_row_groups(B, ks, lo, hi, seed):
    """Teacher heads with windows of 0 rows and empty contexts in the batch: the
    (sequence, head, row group) items with no rows, or no second row group,
    sit between non-empty ones; with contexts of at most 40 keys there are
    fewer key blocks than persistent workgroups."""
    cfg = inputs.scaled(inputs.WORKLOADS["teacher-bf16"], B=B, ctx_lo=lo, ctx_hi=hi, k_choices=ks,
                        models=(inputs.scaled_shape(inputs.TEACHER, vocab=512, hidden=64),))
    _check_all(_case(cfg, seed=seed))


@pytest.mark.parametrize("Hq,Hkv,ks,seed", [(32, 2, (16, 5, 0), 21), (32, 4, (24, 17, 3), 22)])
def test_stream_k_several_row_groups(Hq, Hkv, ks, seed):
    """More than 128 query rows per (sequence, KV head) -- 16 query heads per
    KV head with 16-token windows (256 rows), or 8 with 24-token windows (192
    rows) -- so the stream-K kernel has two 128-row items over the same keys,
    the second partly filled or without rows, and both items' workgroups
    append the same window positions."""
    shape = inputs.ModelShape("wide-groups", Hq=Hq, Hkv=Hkv, D=128, hidden=64, vocab=512)
    cfg = inputs.scaled(inputs.WORKLOADS["teacher-bf16"], B=5, ctx_lo=0, ctx_hi=2500, k_choices=ks,
                        models=(shape,))
    _check_all(_case(cfg, seed=seed))


@pytest.mark.parametrize("lo,hi,seed,weighted", [(480, 540, 31, True), (400, 470, 32, False)])
def test_stream_k_split_near_the_weight_threshold(lo, hi, seed, weighted):
    """64 teacher-head sequences whose key blocks average just above (4256)
    or just below (3660) eight per workgroup: the stream-K split weights its
    spans by XCD and CU slot only from eight blocks per share on, where its
    shortest spans still hold a block, so every workgroup between an item's
    first and last piece has written a partial for the combine."""
    cfg = inputs.scaled(inputs.WORKLOADS["teacher-bf16"], B=64, ctx_lo=lo, ctx_hi=hi,
                        models=(inputs.scaled_shape(inputs.TEACHER, vocab=512, hidden=64),))
    b = _case(cfg, seed=seed)
    blocks = int(sum(-(-(int(L) + int(k)) // 32) for L, k in zip(b.ctx_lens, b.k))) * b.models[0].shape.Hkv
    assert (blocks >= 8 * 512) == weighted, blocks
    _check_all(b)


@pytest.mark.parametrize("ps", [32, 64])
def test_other_page_sizes(ps):
    cfg = inputs.scaled(inputs.WORKLOADS["teacher-bf16"], B=3, ctx_lo=10, ctx_hi=900, page_size=ps,
                        models=(inputs.scaled_shape(inputs.TEACHER, vocab=512, hidden=64),))
    _check_all(_case(cfg, seed=ps))


def test_mixed_windows_and_two_models():
    cfg = inputs.scaled(inputs.WORKLOADS["dual-cache-bf16"], B=10, ctx_lo=0, ctx_hi=700,
                        models=(inputs.scaled_shape(inputs.STUDENT, vocab=512, hidden=64),
                                inputs.scaled_shape(inputs.TEACHER, vocab=512, hidden=64)))
    b = _case(cfg, seed=5)
    _check_all(b, 0)
    _check_all(b, 1)


def test_mixed_windows_repeated_nan_workspace():
    """Regression: short-context, mixed-window teacher-shape batch (items of
    32 rows in 128-row tiles, one block per workgroup, every item split into
    pieces), called repeatedly on a NaN-filled workspace, so that a partial
    read before it is written, or a ring slot refilled before its query
    fragments were read, shows up as a non-finite or wrong row."""
    cfg = inputs.scaled(inputs.WORKLOADS["dual-cache-bf16"], B=10, ctx_lo=0, ctx_hi=700,
                        models=(inputs.scaled_shape(inputs.STUDENT, vocab=512, hidden=64),
                                inputs.scaled_shape(inputs.TEACHER, vocab=512, hidden=64)))
    b = _case(cfg, seed=5)
    mdl = b.models[1]
    seqs = to_np(mdl.seq_ids).astype(np.int64)
    ref, _, _ = parity.oracle_attention(mdl, b, seqs, mdl.shape.D)
    rows = to_np(mdl.rows).astype(np.int64)
    dev = mdl.q.device
    ctx = torch.from_numpy(np.asarray(b.ctx_lens, np.int32)).to(dev)
    cu = torch.from_numpy(np.asarray(b.cu_q, np.int32)).to(dev)
    max_q = int(np.max(np.diff(b.cu_q)))
    n_ws = ops.attn_workspace_size(len(seqs), mdl.shape.Hq, mdl.shape.Hkv, mdl.shape.D, max_q,
                                   mdl.page_table.shape[1], cfg.page_size)
    for rep in range(8):
        ws = torch.full((n_ws,), 0xFF, dtype=torch.uint8, device=dev)   # NaN as float32
        kc, vc = mdl.k_pool.clone(), mdl.v_pool.clone()
        out = ops.verify_attn_paged(mdl.q, mdl.k_new, mdl.v_new, kc, vc, mdl.page_table, ctx, cu,
                                    max_q=max_q, seq_ids=mdl.seq_ids, workspace=ws)
        torch.cuda.synchronize()
        worst = parity.check_attention_rows(out, ref, rows, mdl.q.dtype)
        _say(f"  rep {rep}: worst rel err {worst:.2e}")


def test_head_dim_64_bf16():
    shape = inputs.ModelShape("d64", Hq=8, Hkv=2, D=64, hidden=64, vocab=512)
    cfg = inputs.scaled(inputs.WORKLOADS["teacher-bf16"], B=3, ctx_lo=5, ctx_hi=400, models=(shape,))
    _check_all(_case(cfg, seed=64))


def test_k1_equals_sequential_decode():
    """A k-token window equals k single-token verifies with append."""
    cfg = inputs.scaled(inputs.WORKLOADS["teacher-bf16"], B=2, ctx_lo=200, ctx_hi=700,
                        models=(inputs.scaled_shape(inputs.TEACHER, vocab=512, hidden=64),))
    b = _case(cfg, seed=11)
    mdl = b.models[0]
    out, _, _ = parity.run_gpu_attention(mdl, b)
    kc = mdl.k_pool.clone()
    vc = mdl.v_pool.clone()
    dev = mdl.q.device
    k = int(b.k[0])
    steps = []
    for i in range(k):
        rows = torch.tensor([int(b.cu_q[s]) + i for s in range(b.cfg.B)], device=dev)
        ctx = torch.from_numpy((b.ctx_lens + i).astype(np.int32)).to(dev)
        cu = torch.arange(b.cfg.B + 1, dtype=torch.int32, device=dev)
        o = ops.verify_attn_paged(mdl.q[rows].contiguous(), mdl.k_new[rows].contiguous(),
                                  mdl.v_new[rows].contiguous(), kc, vc, mdl.page_table, ctx, cu,
                                  max_q=1)
        steps.append(o)
    torch.cuda.synchronize()
    dec = torch.stack(steps, 1).reshape(-1, *out.shape[1:])
    g = to_np(out).astype(np.float64)
    d = to_np(dec).astype(np.float64)
    rel = np.linalg.norm(g - d, axis=-1) / np.linalg.norm(d, axis=-1)
    assert rel.max() < 1e-2
    np.testing.assert_array_equal(to_np(kc), to_np(parity.run_gpu_attention(mdl, b)[1]))


def test_eviction_recompute_matches_cached_verify():
    """ctx_len = 0 and the whole prefix + window as rows: the last k rows equal
    the cached verify (Section 3.2.3, preemption recompute)."""
    cfg = inputs.scaled(inputs.WORKLOADS["teacher-bf16"], B=1, ctx_lo=150, ctx_hi=150,
                        models=(inputs.scaled_shape(inputs.TEACHER, vocab=512, hidden=64),))
    b = _case(cfg, seed=12)
    mdl = b.models[0]
    dev = mdl.q.device
    L, k = int(b.ctx_lens[0]), int(b.k[0])
    cached, kc_after, vc_after = parity.run_gpu_attention(mdl, b)
    # rebuild the whole prefix's K/V from the appended cache
    ps = mdl.k_pool.shape[3]
    pos = torch.arange(L + k, device=dev)
    pages = mdl.page_table[0].long()[pos // ps]
    Kall = kc_after[pages, :, :, pos % ps, :].reshape(L + k, mdl.shape.Hkv, mdl.shape.D).contiguous()
    Vall = vc_after[pages, :, :, pos % ps].contiguous()
    qpre = torch.randn(L, mdl.shape.Hq, mdl.shape.D, device=dev).to(mdl.q.dtype)
    qall = torch.cat([qpre, mdl.q[:k]]).contiguous()
    kc = torch.full_like(mdl.k_pool, float("nan"))
    vc = torch.full_like(mdl.v_pool, float("nan"))
    out = ops.verify_attn_paged(qall, Kall, Vall, kc, vc, mdl.page_table,
                                torch.zeros(1, dtype=torch.int32, device=dev),
                                torch.tensor([0, L + k], dtype=torch.int32, device=dev),
                                max_q=L + k)
    torch.cuda.synchronize()
    g = to_np(out[L:]).astype(np.float64)
    c = to_np(cached).astype(np.float64)
    rel = np.linalg.norm(g - c, axis=-1) / np.linalg.norm(c, axis=-1)
    assert rel.max() < 1e-2, rel.max()


def test_full_size_teacher_config_sampled():
    """The full teacher workload (64 sequences, contexts up to 8192) in the
    launch configuration the benchmark times; the oracle checks 3 sequences."""
    b = _case(inputs.WORKLOADS["teacher-bf16"], seed=0, poison=False)
    mdl = b.models[0]
    out, _, _ = parity.run_gpu_attention(mdl, b)
    seqs = [int(np.argmax(b.ctx_lens)), int(np.argmin(b.ctx_lens)), 17]
    ref, rows = parity.oracle_attention_subset(mdl, b, seqs, mdl.shape.D)
    worst = parity.check_attention_rows(out, ref, rows, mdl.q.dtype)
    _say(f"  full teacher config: worst rel err {worst:.2e}")


def test_full_size_long_teacher_config_sampled():
    """The full long-trajectory workload (16 sequences, contexts up to 32768,
    pages shuffled over a 2M-token pool, 16-token windows: two 64-row groups
    per KV head) in the launch configuration the benchmark times; the oracle
    checks the longest and the shortest sequence."""
    b = _case(inputs.WORKLOADS["long-teacher-bf16"], seed=0, poison=False)
    mdl = b.models[0]
    out, _, _ = parity.run_gpu_attention(mdl, b)
    seqs = [int(np.argmax(b.ctx_lens)), int(np.argmin(b.ctx_lens))]
    ref, rows = parity.oracle_attention_subset(mdl, b, seqs, mdl.shape.D)
    worst = parity.check_attention_rows(out, ref, rows, mdl.q.dtype)
    _say(f"  full long-teacher config: worst rel err {worst:.2e}")


def test_full_size_dual_cache_teacher_sampled():
    """The full interleaved dual-cache batch (128 sequences, windows of 1, 4,
    8 or 16, contexts up to 16384): the teacher verifier's call, sampled on
    its longest sequence and on one sequence of each window length."""
    b = _case(inputs.WORKLOADS["dual-cache-bf16"], seed=0, poison=False)
    mdl = b.models[1]
    mine = to_np(mdl.seq_ids).astype(np.int64)
    out, _, _ = parity.run_gpu_attention(mdl, b, seq_ids=mdl.seq_ids)
    seqs = {int(mine[np.argmax(b.ctx_lens[mine])])}
    for k in (1, 4, 8, 16):
        with_k = mine[b.k[mine] == k]
        if len(with_k):
            seqs.add(int(with_k[0]))
    seqs = sorted(seqs)
    ref, rows = parity.oracle_attention_subset(mdl, b, seqs, mdl.shape.D)
    worst = parity.check_attention_rows(out, ref, rows, mdl.q.dtype)
    _say(f"  full dual-cache teacher call, sequences {seqs}: worst rel err {worst:.2e}")


def test_many_sequences_beyond_stream_k_tables():
    """1000 teacher-head sequences: the (sequence, head) items no longer fit
    the stream-K kernel's LDS tables, so the planner takes the register
    kernel for full 64-row groups; both must agree with the oracle."""
    cfg = inputs.scaled(inputs.WORKLOADS["teacher-bf16"], B=1000, ctx_lo=0, ctx_hi=40, pool_tokens=None,
                        models=(inputs.scaled_shape(inputs.TEACHER, vocab=512, hidden=64),))
    _check_all(_case(cfg, seed=11))


def test_stream_k_shares_above_256_blocks():
    """Eight student-head sequences with contexts near 70K tokens: about
    140K key blocks, so each of the stream-K kernel's 512 workgroups streams
    more than 256 blocks and its threads record the page ids of two blocks
    each (the second written at once, the first after the window append's
    loads); the oracle checks the longest and the shortest sequence."""
    base = inputs.WORKLOADS["student-bf16"]
    cfg = inputs.scaled(base, B=8, ctx_lo=68000, ctx_hi=72000,
                        models=(inputs.scaled_shape(base.models[0], vocab=512, hidden=64),))
    b = _case(cfg, seed=13, poison=False)
    mdl = b.models[0]
    blocks = int(sum(-(-(int(L) + int(k)) // 32) for L, k in zip(b.ctx_lens, b.k))) * mdl.shape.Hkv
    assert blocks > 256 * 512, blocks
    out, _, _ = parity.run_gpu_attention(mdl, b)
    seqs = [int(np.argmax(b.ctx_lens)), int(np.argmin(b.ctx_lens))]
    ref, rows = parity.oracle_attention_subset(mdl, b, seqs, mdl.shape.D)
    worst = parity.check_attention_rows(out, ref, rows, mdl.q.dtype)
    _say(f"  {blocks} key blocks: worst rel err {worst:.2e}")
