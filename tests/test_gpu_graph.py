"""One verify step (attention with append, LM head, accept scan, takeover
draw) captured as a HIP graph and replayed, as bench.py times it: every
replay must reproduce the eager step bit for bit.  Between replays the
outputs are overwritten eagerly with a sentinel and other eager work runs,
so a replay that skipped or reused work would show."""
import numpy as np
import pytest
import torch

from paper_2609_36546_amd import inputs, ops
from tests.workload import batch_proposals, to_np

pytestmark = pytest.mark.gpu


class _Step:
    def __init__(self, b, prop):
        cfg, dev = b.cfg, torch.device("cuda")
        self.b, self.K = b, cfg.K
        m = b.models[0]
        self.m = m
        t = lambda a, dt: torch.from_numpy(np.asarray(a, dt)).to(dev)
        self.ctx, self.cu = t(b.ctx_lens, np.int32), t(b.cu_q, np.int32)
        self.driver, self.seq_lens = t(b.driver, np.uint8), t(b.seq_lens, np.int32)
        self.prop = t(prop, np.int32)
        self.max_q = int(b.k.max())
        self.ws_a = torch.empty(ops.attn_workspace_size(cfg.B, m.shape.Hq, m.shape.Hkv, m.shape.D,
                                                        self.max_q, m.page_table.shape[1],
                                                        cfg.page_size), dtype=torch.uint8, device=dev)
        self.ws_l = torch.empty(ops.lmhead_workspace_size(b.T, m.shape.hidden, m.shape.vocab,
                                                          self.K), dtype=torch.uint8, device=dev)
        self.out = torch.empty_like(m.q)
        T, K = b.T, self.K
        self.lm = {"lse": torch.empty(T, device=dev), "logp_prop": torch.empty(T, device=dev),
                   "argmax": torch.empty(T, dtype=torch.int32, device=dev),
                   "topk_idx": torch.empty(T, K, dtype=torch.int32, device=dev),
                   "topk_logp": torch.empty(T, K, device=dev), "entropy": torch.empty(T, device=dev)}
        self.scan = {"n_acc": torch.empty(cfg.B, dtype=torch.int32, device=dev),
                     "event_row": torch.empty(cfg.B, dtype=torch.int32, device=dev),
                     "next_driver": torch.empty(cfg.B, dtype=torch.uint8, device=dev),
                     "finished": torch.empty(cfg.B, dtype=torch.uint8, device=dev),
                     "new_cache_len": torch.empty(cfg.B, dtype=torch.int32, device=dev),
                     "src": torch.empty(T, dtype=torch.uint8, device=dev)}
        self.u = t(b.u_repl, np.float32)
        self.tok = torch.empty(cfg.B, dtype=torch.int32, device=dev)

    def run(self):
        m = self.m
        ops.verify_attn_paged(m.q, m.k_new, m.v_new, m.k_pool, m.v_pool, m.page_table, self.ctx,
                              self.cu, self.max_q, out=self.out, workspace=self.ws_a)
        ops.lmhead_logsoftmax_verify(m.hidden, m.W, self.prop, self.K, outs=self.lm,
                                     workspace=self.ws_l)
        ops.accept_scan(self.cu, self.prop, self.lm["topk_idx"], self.K, self.driver, self.ctx,
                        self.seq_lens, self.b.eos_id, self.b.max_len, outs=self.scan)
        ops.sample_takeover(m.hidden, m.W, self.K, self.ws_l, self.cu, self.driver,
                            self.scan["event_row"], self.u, self.b.eos_id, self.scan["finished"],
                            token=self.tok)

    def outputs(self):
        o = {"out": self.out, "tok": self.tok, "k_pool": self.m.k_pool, "v_pool": self.m.v_pool}
        o.update({f"lm_{k}": v for k, v in self.lm.items()})
        o.update({f"scan_{k}": v for k, v in self.scan.items()})
        return {k: v.clone() for k, v in o.items()}

    def scramble(self):
        for t in [self.out, self.tok] + list(self.lm.values()) + list(self.scan.values()):
            t.fill_(7 if t.dtype in (torch.int32, torch.uint8) else float("nan"))


def test_graph_replays_equal_eager_step():
    cfg = inputs.scaled(inputs.WORKLOADS["teacher-bf16"], B=8, ctx_lo=100, ctx_hi=2000,
                        models=(inputs.scaled_shape(inputs.TEACHER, vocab=20000),))
    print(f"[graph] {cfg.name} B={cfg.B} V=20000", flush=True)
    b = inputs.make_batch(cfg, seed=5, device="cuda")
    st = _Step(b, batch_proposals(b))
    st.run()
    torch.cuda.synchronize()
    ref = st.outputs()
    assert int((to_np(ref["scan_event_row"]) >= 0).sum()) > 0     # some takeovers happen
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        st.run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        st.run()
    x = torch.randn(512, 512, device="cuda")
    for rep in range(4):
        st.scramble()                       # eager work between replays
        y = x @ x
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = st.outputs()
        for k in ref:
            a, r = to_np(got[k]), to_np(ref[k])
            np.testing.assert_array_equal(np.isnan(a) if a.dtype.kind == "f" else a,
                                          np.isnan(r) if r.dtype.kind == "f" else r, err_msg=k)
            if a.dtype.kind == "f":
                np.testing.assert_array_equal(a[~np.isnan(a)], r[~np.isnan(r)], err_msg=f"{k} replay {rep}")
        del y
