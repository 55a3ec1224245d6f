"""verify_attn_paged_noalloc (the allocation-free attention entry point)
against verify_attn_paged with a caller workspace, through the C ABI.

Both run the same kernels and split plan, so the outputs and the appended
caches must be bit-identical (stricter than the attention parity bound).
Two calls in a row on the same GPU: the full teacher workload, then a small
batch, which reuses the scratch with the first call's partials still in it
(nothing in it may need to start at zero).  A call whose partials exceed the
scratch is rejected on the host before any launch.
"""
import numpy as np
import pytest
import torch

from paper_2609_36546_amd import inputs, ops
from tests.workload import to_np

pytestmark = pytest.mark.gpu


def _both(b, mi=0):
    m = b.models[mi]
    dev = m.q.device
    ctx = torch.from_numpy(b.ctx_lens).to(dev)
    cu = torch.from_numpy(b.cu_q).to(dev)
    max_q = int(b.k.max())
    need = ops.attn_workspace_size(m.seq_ids.shape[0], m.shape.Hq, m.shape.Hkv, m.shape.D, max_q,
                                   m.page_table.shape[1], b.cfg.page_size)
    print(f"[noalloc] {b.cfg.name} B={b.cfg.B}: workspace {need} bytes", flush=True)
    assert 0 < need <= ops.NOALLOC_SCRATCH_BYTES
    kc1, vc1 = m.k_pool.clone(), m.v_pool.clone()
    ref = ops.verify_attn_paged(m.q, m.k_new, m.v_new, kc1, vc1, m.page_table, ctx, cu, max_q,
                                seq_ids=m.seq_ids)
    kc2, vc2 = m.k_pool.clone(), m.v_pool.clone()
    out = torch.full_like(m.q, float("nan"))
    ops.verify_attn_paged_noalloc(m.q, m.k_new, m.v_new, kc2, vc2, m.page_table, ctx, cu, max_q,
                                  seq_ids=m.seq_ids, out=out)
    torch.cuda.synchronize()
    rows = m.rows.long()
    bits = lambda t: t.view(torch.int16 if t.element_size() == 2 else torch.int32)
    # bit patterns, so that the NaN poison of unused pool slots compares equal
    assert torch.equal(bits(out[rows]), bits(ref[rows]))
    assert torch.equal(bits(kc1), bits(kc2)) and torch.equal(bits(vc1), bits(vc2))
    return need


def test_noalloc_equals_workspace_call_twice_then_smaller():
    big = inputs.make_batch(inputs.WORKLOADS["teacher-bf16"], seed=0, device="cuda", poison=False)
    n1 = _both(big)
    small_cfg = inputs.scaled(inputs.WORKLOADS["student-bf16"], B=5, ctx_lo=3, ctx_hi=700,
                              models=(inputs.scaled_shape(inputs.STUDENT, vocab=512, hidden=64),))
    small = inputs.make_batch(small_cfg, seed=3, device="cuda", poison=True)
    n2 = _both(small)
    assert n2 < n1


def test_noalloc_rejects_a_call_above_the_scratch_limit():
    b = inputs.make_batch(inputs.scaled(inputs.WORKLOADS["teacher-bf16"], B=4, ctx_lo=10, ctx_hi=50,
                                        models=(inputs.scaled_shape(inputs.TEACHER, vocab=512,
                                                                    hidden=64),)),
                          seed=1, device="cuda", poison=False)
    m = b.models[0]
    dev = m.q.device
    # a page table wide enough that the split plan's partials exceed the scratch
    wide = torch.zeros(b.cfg.B, 200000, dtype=torch.int32, device=dev)
    wide[:, :m.page_table.shape[1]] = m.page_table
    assert ops.attn_workspace_size(b.cfg.B, 32, 4, 128, 8, 200000, 16) > ops.NOALLOC_SCRATCH_BYTES
    with pytest.raises(ops.IpdvError) as e:
        ops.verify_attn_paged_noalloc(m.q, m.k_new, m.v_new, m.k_pool.clone(), m.v_pool.clone(),
                                      wide, torch.from_numpy(b.ctx_lens).to(dev),
                                      torch.from_numpy(b.cu_q).to(dev), int(b.k.max()))
    assert e.value.status == -2 and "scratch" in str(e.value)
