"""The C-ABI library loads and exports every symbol include/ipdv.h declares;
host-side validation returns the documented statuses (no GPU calls)."""
import ctypes
import os
import re

import pytest

from paper_2609_36546_amd import ops

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ipdv.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b([a-z_][a-z0-9_]*)\s*\(", text)) -
                  {"sizeof", "defined", "if", "extern"})


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("verify_attn_paged", "lmhead_logsoftmax_verify", "accept_scan", "accept_scan_rule",
              "sample_takeover"):
        assert n in names


def test_library_exports_every_declared_symbol():
    L = ops.lib()
    for n in declared_functions():
        assert hasattr(L, n), f"libipdv.so does not export {n}"
    assert "gfx950" in ops.version()


def _attn(**kw):
    args = dict(q=1, k_new=1, v_new=1, k_cache=1, v_cache=1, page_table=1, maxp=4, ctx=1, cu=1,
                seq_ids=None, n_seq=2, max_q=4, out=1, Hq=4, Hkv=2, D=64, ps=16, P=8,
                scale=0.125, dtype=ops.IPDV_BF16, ws=1, wsb=1 << 30, stream=None)
    args.update(kw)
    a = args
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    return ops.lib().verify_attn_paged(
        vp(a["q"]), vp(a["k_new"]), vp(a["v_new"]), vp(a["k_cache"]), vp(a["v_cache"]),
        vp(a["page_table"]), a["maxp"], vp(a["ctx"]), vp(a["cu"]), vp(a["seq_ids"]), a["n_seq"],
        a["max_q"], vp(a["out"]), a["Hq"], a["Hkv"], a["D"], a["ps"], a["P"], a["scale"],
        a["dtype"], vp(a["ws"]), a["wsb"], vp(a["stream"]))


@pytest.mark.parametrize("kw,status", [
    (dict(D=96), -2), (dict(ps=8), -2), (dict(ps=48), -2), (dict(Hq=6, Hkv=4), -1),
    (dict(q=None), -1), (dict(max_q=0), -1), (dict(n_seq=-1), -1), (dict(dtype=7), -2),
    (dict(wsb=10), -3), (dict(ws=None), -3), (dict(scale=float("inf")), -1), (dict(scale=-0.1), -1),
    (dict(P=0), -1), (dict(maxp=0), -1), (dict(dtype=ops.IPDV_F32, D=128), -2)])
def test_attention_argument_errors(kw, status):
    assert _attn(**kw) == status
    assert ops.lib().ipdv_last_error().decode() != ""


def test_attention_empty_batch_is_ok_without_gpu():
    assert _attn(n_seq=0, q=None) == 0


def test_workspace_size_queries():
    assert ops.attn_workspace_size(64, 32, 4, 128, 8, 513, 16) > 0
    assert ops.attn_workspace_size(64, 32, 4, 96, 8, 513, 16) == 0
    assert ops.lmhead_workspace_size(512, 2048, 151936, 16) > 0
    assert ops.lmhead_workspace_size(512, 2048, 151936, 33) == 0
    assert ops.lmhead_workspace_size(8, 100, 1024, 16) == 0


def _ws(which, args, n=None):
    arr = (ctypes.c_int32 * max(len(args), 1))(*args)
    return ops.lib().ipdv_workspace_size(which, arr, len(args) if n is None else n)


def test_workspace_size_dispatcher_matches_the_typed_queries():
    for a in [(64, 32, 4, 128, 8, 513, 16), (32, 16, 8, 128, 8, 257, 16), (3, 4, 2, 64, 4, 9, 32),
              (64, 32, 4, 96, 8, 513, 16)]:
        assert _ws(0, a) == ops.attn_workspace_size(*a)
    for a in [(512, 2048, 151936, 16), (8, 256, 1024, 32), (512, 2048, 151936, 33)]:
        assert _ws(1, a) == ops.lmhead_workspace_size(*a)
    assert _ws(0, (64, 32, 4, 128, 8, 513)) == 0          # wrong count
    assert _ws(1, (512, 2048, 151936, 16), n=5) == 0
    assert _ws(2, (512, 2048, 151936, 16)) == 0          # unknown kind
    assert ops.lib().ipdv_workspace_size(1, None, 4) == 0
    assert "shape" in ops.lib().ipdv_last_error().decode() or \
        "NULL" in ops.lib().ipdv_last_error().decode()


def _lm(**kw):
    a = dict(h=1, W=1, prop=1, rows=None, M=8, Hd=256, V=1024, K=16, lse=1, lp=1, am=1, ti=1, tl=1,
             ent=None, dtype=ops.IPDV_F32, ws=1, wsb=1 << 30)
    a.update(kw)
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    return ops.lib().lmhead_logsoftmax_verify(
        vp(a["h"]), vp(a["W"]), vp(a["prop"]), vp(a["rows"]), a["M"], a["Hd"], a["V"], a["K"],
        vp(a["lse"]), vp(a["lp"]), vp(a["am"]), vp(a["ti"]), vp(a["tl"]), vp(a["ent"]), a["dtype"],
        vp(a["ws"]), a["wsb"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(K=0), -1), (dict(K=33), -1), (dict(K=17, V=16), -1), (dict(Hd=100), -2),
    (dict(M=-1), -1), (dict(V=0), -1), (dict(W=None), -1), (dict(dtype=3), -2),
    (dict(wsb=0), -3)])
def test_lmhead_argument_errors(kw, status):
    assert _lm(**kw) == status


def test_lmhead_empty_is_ok_without_gpu():
    assert _lm(M=0, h=None) == 0


def test_scan_argument_errors():
    L = ops.lib()
    vp = ctypes.c_void_p
    args = [vp(1), vp(1), vp(1), 4, vp(1), vp(1), vp(1), 0, 100, 3] + [vp(1)] * 6 + [None]
    bad_K = list(args)
    bad_K[3] = 33
    assert L.accept_scan(*bad_K) == -1
    bad_B = list(args)
    bad_B[9] = -2
    assert L.accept_scan(*bad_B) == -1
    null_out = list(args)
    null_out[12] = None
    assert L.accept_scan(*null_out) == -1
    empty = list(args)
    empty[9] = 0
    assert L.accept_scan(*empty) == 0


def test_scan_rule_argument_errors():
    L = ops.lib()
    vp = ctypes.c_void_p

    def args(take=0, hand=0, ent=vp(1), topk=vp(1), B=3):
        return ([vp(1), vp(1), topk, 4, vp(1), vp(1), vp(1), 0, 100, B, take, hand, ent,
                 0.5, 0.5] + [vp(1)] * 6 + [None])
    assert L.accept_scan_rule(*args(take=2)) == -1            # unknown takeover rule
    assert L.accept_scan_rule(*args(hand=3)) == -1            # unknown handback rule
    assert L.accept_scan_rule(*args(take=-1)) == -1
    assert L.accept_scan_rule(*args(take=1, ent=None)) == -1  # entropy rule without ent
    assert L.accept_scan_rule(*args(hand=2, ent=None)) == -1
    assert L.accept_scan_rule(*args(topk=None)) == -1         # coverage rule, K > 0, no top-K
    # rules are validated before the empty-batch shortcut
    assert L.accept_scan_rule(*args(take=5, B=0)) == -1
    assert L.accept_scan_rule(*args(take=1, hand=2, B=0)) == 0


def test_lmhead_vocab_limit():
    assert _lm(V=262145, K=16) == -2


def _sample(**kw):
    args = dict(hidden=1, W=1, M=8, Hd=256, V=1024, K=16, ws=1, wsb=1 << 30, seq_ids=None, n_seq=2,
                cu=1, driver=1, ev=1, row_local=None, u=1, eos=1023, token=1, fin=1,
                dtype=ops.IPDV_BF16)
    args.update(kw)
    a = args
    vp = lambda x: None if x is None else ctypes.c_void_p(x)
    return ops.lib().sample_takeover(
        vp(a["hidden"]), vp(a["W"]), a["M"], a["Hd"], a["V"], a["K"], vp(a["ws"]), a["wsb"],
        vp(a["seq_ids"]), a["n_seq"], vp(a["cu"]), vp(a["driver"]), vp(a["ev"]),
        vp(a["row_local"]), vp(a["u"]), a["eos"], vp(a["token"]), vp(a["fin"]), a["dtype"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(u=None), -1), (dict(token=None), -1), (dict(W=None), -1), (dict(n_seq=-1), -1),
    (dict(K=33), -1), (dict(Hd=100), -2), (dict(dtype=5), -2), (dict(wsb=10), -3), (dict(ws=None), -3)])
def test_sample_argument_errors(kw, status):
    assert _sample(**kw) == status
    assert ops.lib().ipdv_last_error().decode() != ""


def test_sample_empty_batch_is_ok_without_gpu():
    assert _sample(n_seq=0, u=None, token=None) == 0


def test_gather_and_kl_argument_errors():
    L = ops.lib()
    vp = ctypes.c_void_p
    # lmhead_logp_gather(hidden, W, M, Hd, V, lse, idx, n_idx, logp, dtype, stream)
    g = [vp(1), vp(1), 4, 128, 1000, vp(1), vp(1), 16, vp(1), 1, None]
    bad = list(g); bad[7] = 65
    assert L.lmhead_logp_gather(*bad) == -1           # n_idx above IPDV_MAX_GATHER
    bad = list(g); bad[3] = 100
    assert L.lmhead_logp_gather(*bad) == -2           # Hd not a multiple of 64
    bad = list(g); bad[6] = None
    assert L.lmhead_logp_gather(*bad) == -1
    bad = list(g); bad[9] = 7
    assert L.lmhead_logp_gather(*bad) == -2          # unknown dtype
    bad = list(g); bad[9] = 0x10
    assert L.lmhead_logp_gather(*bad) == -2          # tiled W is bf16 only
    empty = list(g); empty[7] = 0
    assert L.lmhead_logp_gather(*empty) == 0
    # source_split_kl(M, K, s_idx, s_logp, s_at_t, t_idx, t_logp, t_at_s, src, support,
    #                 loss_mode, kl_rev, kl_fwd, loss, overlap, cu, B, seq_loss, t_ratio, stream)
    k = [8, 16] + [vp(1)] * 7 + [0, 0] + [vp(1)] * 4 + [vp(1), 3, vp(1), vp(1), None]
    bad = list(k); bad[1] = 33
    assert L.source_split_kl(*bad) == -1
    bad = list(k); bad[1] = 0
    assert L.source_split_kl(*bad) == -1
    bad = list(k); bad[9] = 4
    assert L.source_split_kl(*bad) == -1              # unknown support
    bad = list(k); bad[10] = -1
    assert L.source_split_kl(*bad) == -1              # unknown loss mode
    bad = list(k); bad[8] = None
    assert L.source_split_kl(*bad) == -1              # loss without src
    bad = list(k); bad[13] = None
    assert L.source_split_kl(*bad) == -1              # segments without the row loss
    bad = list(k); bad[16] = -1
    assert L.source_split_kl(*bad) == -1
    empty = list(k); empty[0] = 0; empty[16] = 0
    assert L.source_split_kl(*empty) == 0


def test_binding_and_oracle_constants_match_the_header():
    import oracle
    defs = dict((m.group(1), int(m.group(2))) for m in
                re.finditer(r"#define\s+(IPDV_\w+)\s+(-?\d+)", open(HEADER).read()))
    pairs = {"TAKE_COVERAGE": "IPDV_TAKE_COVERAGE", "TAKE_ENTROPY": "IPDV_TAKE_ENTROPY",
             "HAND_COVERAGE": "IPDV_HAND_COVERAGE", "HAND_FIXED_ONE": "IPDV_HAND_FIXED_ONE",
             "HAND_ENTROPY": "IPDV_HAND_ENTROPY", "SUPPORT_UNION": "IPDV_SUPPORT_UNION",
             "SUPPORT_STUDENT": "IPDV_SUPPORT_STUDENT", "SUPPORT_TEACHER": "IPDV_SUPPORT_TEACHER",
             "SUPPORT_INTERSECTION": "IPDV_SUPPORT_INTERSECTION",
             "LOSS_IPD_SPLIT": "IPDV_LOSS_IPD_SPLIT", "LOSS_PURE_REVERSE": "IPDV_LOSS_PURE_REVERSE",
             "LOSS_PURE_FORWARD": "IPDV_LOSS_PURE_FORWARD",
             "LOSS_INVERSE_SPLIT": "IPDV_LOSS_INVERSE_SPLIT"}
    for name, macro in pairs.items():
        assert getattr(ops, name) == defs[macro], name
        assert getattr(oracle, name) == defs[macro], name
    for name, macro in (("DRIVER_S", "IPDV_DRIVER_S"), ("DRIVER_T", "IPDV_DRIVER_T"),
                        ("SRC_S", "IPDV_SRC_S"), ("SRC_T", "IPDV_SRC_T"),
                        ("SRC_DISCARDED", "IPDV_SRC_DISCARDED")):
        assert getattr(oracle, name) == defs[macro], name
    m = re.search(r"#define\s+IPDV_NOALLOC_SCRATCH_BYTES\s+\((\d+)u\s*<<\s*(\d+)\)", open(HEADER).read())
    assert ops.NOALLOC_SCRATCH_BYTES == int(m.group(1)) << int(m.group(2))


def test_tiled_w_argument_errors():
    L = ops.lib()
    vp = ctypes.c_void_p
    L.ipdv_lmhead_packed_w_size.argtypes = [ctypes.c_int, ctypes.c_int]
    L.ipdv_lmhead_packed_w_size.restype = ctypes.c_size_t
    assert L.ipdv_lmhead_packed_w_size(151936, 2048) == 151936 * 2048 * 2
    assert L.ipdv_lmhead_packed_w_size(100, 64) == 112 * 64 * 2     # rows padded to 16
    assert L.ipdv_lmhead_packed_w_size(100, 100) == 0                # Hd not a multiple of 64
    assert L.lmhead_pack_w(vp(1), 100, 64, vp(2), 0, None) == -2     # fp32: unsupported
    assert L.lmhead_pack_w(None, 100, 64, vp(2), 1, None) == -1
    assert L.lmhead_pack_w(vp(1), 100, 64, vp(1), 1, None) == -1     # aliasing
    assert L.lmhead_pack_w(vp(1), 0, 64, vp(2), 1, None) == -1       # V < 1
    # fp32 with the tiled flag is refused by every call that reads W
    args = dict(M=4, Hd=64, V=100, K=4)
    st = L.lmhead_logsoftmax_verify(vp(1), vp(1), vp(1), None, 4, 64, 100, 4, vp(1), vp(1),
                                    vp(1), vp(1), vp(1), None, 0x10, vp(1), 1 << 30, None)
    assert st == -2
    st = L.lmhead_sample(vp(1), vp(1), 4, 64, 100, 4, vp(1), 1 << 30, vp(1), vp(1), 0x10, None)
    assert st == -2


def _table(seed=0, B=6, ps=16, maxp=12):
    """A valid page table: every sequence's pages distinct, drawn from a pool."""
    import numpy as np
    rng = np.random.default_rng(seed)
    ctx = rng.integers(0, maxp * ps - 20, size=B).astype(np.int32)
    k = rng.integers(0, 9, size=B).astype(np.int32)
    cu = np.concatenate([[0], np.cumsum(k)]).astype(np.int32)
    P = B * maxp + 3
    pt = rng.permutation(P)[:B * maxp].reshape(B, maxp).astype(np.int32)
    return pt, ctx, cu, P


def test_page_table_check_accepts_valid_tables():
    import numpy as np
    for seed in range(5):
        pt, ctx, cu, P = _table(seed)
        ops.check_page_table(pt, ctx, cu, max_q=8, page_size=16, num_pages=P)
        ops.check_page_table(pt, ctx, cu, max_q=8, page_size=16, num_pages=P,
                             seq_ids=np.array([4, 1, 2], np.int32))
    # entries past a sequence's need are never read: any value is accepted
    pt, ctx, cu, P = _table(7)
    need = -(-(ctx + np.diff(cu)) // 16)
    for b in range(len(ctx)):
        pt[b, need[b]:] = -5
    ops.check_page_table(pt, ctx, cu, max_q=8, page_size=16, num_pages=P)
    # a shared prefix page that no window writes is fine
    pt, ctx, cu, P = _table(8)
    ctx[:2] = 40
    cu = np.concatenate([[0], np.cumsum(np.diff(cu))]).astype(np.int32)
    pt[1, 0] = pt[0, 0]
    ops.check_page_table(pt, ctx, cu, max_q=8, page_size=16, num_pages=P)


def test_page_table_check_names_each_violation():
    import numpy as np

    def expect(fragment, pt, ctx, cu, P, seq, **kw):
        with pytest.raises(ops.IpdvError, match=fragment):
            ops.check_page_table(pt, ctx, cu, page_size=16, num_pages=P, **kw)
        bad = ctypes.c_int32(-7)
        p = lambda a: None if a is None else np.ascontiguousarray(a, np.int32).ctypes.data_as(ctypes.c_void_p)
        sid = kw.get("seq_ids")
        n = len(ctx) if sid is None else len(sid)
        assert ops.lib().ipdv_check_page_table(
            p(pt), len(ctx), pt.shape[1], p(ctx), p(cu), p(sid), n, kw["max_q"], 16, P,
            ctypes.byref(bad)) == -1
        assert bad.value == seq

    pt, ctx, cu, P = _table(1)
    k = np.diff(cu)
    b = int(np.argmax(ctx + k))
    x = pt.copy()
    x[b, (ctx[b] + k[b] - 1) // 16] = P                  # page id out of range
    expect("not in", x, ctx, cu, P, b, max_q=8)
    x = pt.copy()
    x[b, 0] = -1
    expect("not in", x, ctx, cu, P, b, max_q=8)
    c = ctx.copy()
    c[2] = -3                                            # negative context
    expect("ctx_len", pt, c, cu, P, 2, max_q=8)
    c = ctx.copy()
    c[3] = 12 * 16                                       # does not fit the table
    expect("do not fit", pt, c, cu, P, 3, max_q=8)
    expect("exceeds max_q", pt, ctx, cu, P, int(np.argmax(k)), max_q=int(k.max()) - 1)
    u = cu.copy()
    u[0] = 1
    expect("cu_q", pt, ctx, u, P, 0, max_q=8)
    # two windows writing one page, and a window page read by another sequence
    c = ctx.copy()
    c[0], c[1] = 33, 50
    u = np.concatenate([[0], np.cumsum(np.r_[4, 4, k[2:]])]).astype(np.int32)
    x = pt.copy()
    x[1, 3] = x[0, 2]
    expect("written by the windows", x, c, u, P, 1, max_q=8)
    x = pt.copy()
    x[1, 0] = x[0, 2]
    expect("read by sequence", x, c, u, P, 1, max_q=8)
    expect("listed twice", pt, ctx, cu, P, 2, max_q=8, seq_ids=np.array([2, 2], np.int32))
    expect("seq_ids", pt, ctx, cu, P, -1, max_q=8, seq_ids=np.array([0, 9], np.int32))


def test_noalloc_attention_rejects_calls_above_its_scratch_on_the_host():
    """The allocation-free entry point checks its arguments like
    verify_attn_paged and refuses a call whose split-KV partials exceed its
    scratch, before any HIP call (dummy pointers: nothing is launched)."""
    vp = ctypes.c_void_p
    L = ops.lib()

    def call(maxp, n_seq=4, D=128, q=1):
        return L.verify_attn_paged_noalloc(vp(q), vp(1), vp(1), vp(1), vp(1), vp(1), maxp, vp(1),
                                           vp(1), None, n_seq, 8, vp(1), 32, 4, D, 16, 8, 0.088,
                                           ops.IPDV_BF16, None)
    assert ops.attn_workspace_size(4, 32, 4, 128, 8, 200000, 16) > ops.NOALLOC_SCRATCH_BYTES
    assert call(200000) == -2
    assert "scratch" in L.ipdv_last_error().decode()
    assert call(100, D=96) == -2                 # the same argument checks as verify_attn_paged
    assert call(100, q=None) == -1
    assert call(100, n_seq=0, q=None) == 0       # nothing to do
