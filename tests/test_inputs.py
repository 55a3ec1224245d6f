"""Structure of the seeded synthetic batches (host logic, CPU only)."""
import numpy as np
import torch

from paper_2609_36546_amd import inputs
from tests.workload import to_np


def small(name, **kw):
    return inputs.scaled(inputs.WORKLOADS[name], **kw)


def test_tiny_config_structure_and_poison():
    b = inputs.make_batch(inputs.WORKLOADS["tiny-f32"], seed=0)
    cfg = b.cfg
    assert b.T == 8 and list(b.k) == [4, 4] and list(b.ctx_lens) == [128, 128]
    assert list(b.driver) == [inputs.DRIVER_S, inputs.DRIVER_T]
    m = b.models[0]
    pt = to_np(m.page_table)
    ps = cfg.page_size
    used = []
    for s in range(cfg.B):
        need = -(-(b.ctx_lens[s] + b.k[s]) // ps)
        used.extend(pt[s, :need])
        assert np.all(pt[s, need:] == m.poison_page)
    assert len(set(used)) == len(used) and m.poison_page not in used
    kp = to_np(m.k_pool)
    assert np.all(np.isnan(kp[m.poison_page]))
    # cached slots are finite, slots at and after L are poison
    L = b.ctx_lens[0]
    page = pt[0, L // ps]
    assert np.all(np.isnan(kp[page, :, :, L % ps, :]))
    assert np.all(np.isfinite(kp[pt[0, 0], :, :, 0, :]))


def test_seeded_and_reproducible():
    a = inputs.make_batch(small("teacher-bf16", B=4, ctx_lo=20, ctx_hi=90, models=(inputs.TINY,)), seed=5)
    b = inputs.make_batch(small("teacher-bf16", B=4, ctx_lo=20, ctx_hi=90, models=(inputs.TINY,)), seed=5)
    assert np.array_equal(a.ctx_lens, b.ctx_lens)
    assert torch.equal(a.models[0].q, b.models[0].q)
    assert torch.equal(a.models[0].W, b.models[0].W)
    assert np.array_equal(a.u_tok, b.u_tok)


def test_dual_config_split_and_row_maps():
    cfg = small("dual-cache-bf16", B=16, ctx_lo=16, ctx_hi=64,
                models=(inputs.scaled_shape(inputs.STUDENT, vocab=64, hidden=32),
                        inputs.scaled_shape(inputs.TEACHER, vocab=64, hidden=32)))
    b = inputs.make_batch(cfg, seed=0)
    assert int((b.driver == inputs.DRIVER_T).sum()) == 8
    rows_seen = []
    for mi, m in enumerate(b.models):
        seqs = to_np(m.seq_ids)
        assert np.all(b.verifier[seqs] == mi)
        # the verifier is the counterpart of the driver: student verifies driver T
        assert np.all(b.driver[seqs] == (inputs.DRIVER_T if mi == 0 else inputs.DRIVER_S))
        rows = to_np(m.rows)
        assert len(rows) == m.hidden.shape[0]
        rows_seen.extend(rows)
    assert sorted(rows_seen) == list(range(b.T))
    assert set(np.unique(b.k)) <= {1, 4, 8, 16}
