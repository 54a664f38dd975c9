"""The boundary contract on the GPU, through the C ABI.

* Stateless entry points: the content of the workspace before a call does
  not matter (nothing is kept between calls), so a workspace filled with
  arbitrary bytes before every call gives results identical to a zeroed one.
* Caller-supplied topologies and node tokens are checked before any entry
  becomes an address: out-of-range entries set TSB_REQ_BAD_TREE /
  TSB_REQ_BAD_TOKEN for their own request (n_acc = bonus = -1) and leave
  every other request bit-identical; replay skips malformed parents.
"""
import numpy as np
import pytest
import torch

import workloads as W
import paper_2609_33652_amd as tsb

pytestmark = pytest.mark.gpu

OUT_KEYS = ("draft_lse", "topk_tok", "topk_lp", "parent", "depth", "rank", "n_children", "first_child", "score",
            "n_nodes", "plan_margin", "node_tok", "n_acc", "acc_node", "acc_tok", "bonus", "req_status",
            "target_lse", "trace", "pool_tok")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tsb.load()


def _same(a, b):
    if a is None or b is None:
        return a is None and b is None
    if a.dtype.is_floating_point:
        return torch.equal(a.nan_to_num(7.0), b.nan_to_num(7.0))
    return torch.equal(a, b)


def _inputs(cfg, P):
    base, sigma = W.base_rows(cfg, 0)
    draft = W.draft_from_base(cfg, base)
    dep = torch.ones(cfg["R"], cfg["B"] + 1, dtype=torch.int64)
    target = W.target_from_base(cfg, base, sigma, dep)
    trans = W.transitions(cfg, P)
    return draft.cuda(), target.cuda(), trans.cuda()


@pytest.mark.parametrize("kind", ["step", "step_first", "pool_step"])
def test_workspace_content_does_not_matter(kind):
    cfg = W.config(2, R=4, V=20000, D=6, B=24, K=5, name="stateless")
    P = 16
    draft, target, trans = _inputs(cfg, P)
    c = tsb.make_config(cfg["R"], cfg["D"], cfg["V"], cfg["B"], cfg["K"], cfg["T"], cfg["dtype"], 77)
    clean = tsb.Round(c, "cuda", target_lse=True, trace=True, pool=P)
    dirty = tsb.Round(c, "cuda", target_lse=True, trace=True, pool=P)
    fills = (0xA5, 0xFF, 0x5A, 0x01)
    for s, fill in enumerate(fills):
        clean.ws.zero_()
        dirty.ws.fill_(fill)
        for rnd in (clean, dirty):
            if kind == "pool_step":
                rnd.pool_step(draft, trans, target, s)
            else:
                getattr(rnd, kind)(draft, target, s)
        a, b = clean.host(), dirty.host()
        for k in OUT_KEYS:
            if kind == "step_first" and k in ("trace", "target_lse"):
                continue  # the Naive walk writes neither
            if kind != "pool_step" and k == "pool_tok":
                continue  # written by the pool round only (an unwritten output buffer)
            assert _same(a[k], b[k]), (kind, s, hex(fill), k)
        assert int((a["req_status"] & tsb.REQ_WALK_TIMEOUT).sum()) == 0


def test_workspace_reused_across_entry_points_without_clearing():
    """One workspace serves the RRS walk, the Naive walk and the pool walk in turn, never cleared by the caller:
    every call equals the same call on a fresh zeroed workspace."""
    cfg = W.config(2, R=3, V=12000, D=5, B=20, K=4, name="shared")
    P = 16
    draft, target, trans = _inputs(cfg, P)
    c = tsb.make_config(cfg["R"], cfg["D"], cfg["V"], cfg["B"], cfg["K"], cfg["T"], cfg["dtype"], 5)
    shared = tsb.Round(c, "cuda", target_lse=True, trace=True, pool=P)
    shared.ws.fill_(0xC3)
    seq = ["step", "step_first", "pool_step", "step", "pool_step", "step_first"]
    for s, kind in enumerate(seq):
        fresh = tsb.Round(c, "cuda", target_lse=True, trace=True, pool=P)
        fresh.ws.zero_()
        for rnd in (shared, fresh):
            if kind == "pool_step":
                rnd.pool_step(draft, trans, target, s)
            else:
                getattr(rnd, kind)(draft, target, s)
        a, b = fresh.host(), shared.host()
        keys = ("n_acc", "acc_node", "acc_tok", "bonus", "req_status", "node_tok")
        for k in keys + (() if kind == "step_first" else ("trace",)):  # the Naive walk writes no trace
            assert _same(a[k], b[k]), (kind, s, k)


def _planned(cfg, seed, draft):
    c = tsb.make_config(cfg["R"], cfg["D"], cfg["V"], cfg["B"], cfg["K"], cfg["T"], cfg["dtype"], seed)
    rnd = tsb.Round(c, "cuda", target_lse=True, trace=True)
    rnd.plan(draft)
    rnd.replay(draft, 0)
    return c, rnd


def _corrupt(tree, tok, D, B, V):
    """Requests 1..5 get one out-of-range entry each at the root (which has children); request 0 stays clean.
    Returns the set of requests whose walk must flag BAD_TREE, and (request -> expected bit) for tokens."""
    t = {k: v.clone() for k, v in tree.items()}
    n = t["n_nodes"].clone()
    assert (t["n_children"][:, 0] > 0).all()
    t["n_children"][1, 0] = tsb.MAX_K + 8           # more children than a node may have
    t["first_child"][2, 0] = int(n[2])               # children beyond n_nodes
    t["first_child"][3, 0] = 0                       # a child index not after its parent (a cycle)
    t["depth"][4, 0] = D                             # a depth without a draft row
    t["n_nodes"][5] = B + 2                          # more nodes than the budget holds
    return t


@pytest.mark.parametrize("entry", ["verify", "verify_naive", "pool_verify", "replay"])
def test_malformed_tree_is_flagged_not_used(entry):
    cfg = dict(name="malformed", R=6, V=3000, D=4, B=12, K=3, T=1.0, dtype="f32")
    rng = np.random.default_rng(8)
    draft = torch.from_numpy((rng.standard_normal((6, 4, 3000)) * 2).astype(np.float32)).cuda()
    target = torch.from_numpy((rng.standard_normal((6, 13, 3000)) * 2).astype(np.float32)).cuda()
    P = 8
    trans = torch.from_numpy(rng.standard_normal((6, 3, P, P)).astype(np.float32)).cuda()
    c = tsb.make_config(6, 4, 3000, 12, 3, 1.0, "f32", 3)
    ref = tsb.Round(c, "cuda", target_lse=True, trace=True, pool=P)
    bad = tsb.Round(c, "cuda", target_lse=True, trace=True, pool=P)
    if entry == "pool_verify":
        ref.pool_plan(draft, trans)
        ref.pool_replay(draft, trans, 0)
    else:
        ref.plan(draft)
        ref.replay(draft, 0)
    clean_tree = {k: v.clone() for k, v in ref.tree.items()}
    clean_tok = ref.node_tok.clone()
    bad.load_tree(_corrupt(clean_tree, clean_tok, 4, 12, 3000))
    bad.node_tok.copy_(clean_tok)
    if entry == "pool_verify":
        bad.pool_tok.copy_(ref.pool_tok)
        ref.req_status.zero_()
        bad.req_status.zero_()
        ref.pool_verify(draft, trans, target, 0)
        bad.pool_verify(draft, trans, target, 0)
    elif entry == "verify":
        bad.draft_lse.copy_(ref.draft_lse)
        ref.req_status.zero_()
        bad.req_status.zero_()
        ref.verify(draft, target, 0)
        bad.verify(draft, target, 0)
    elif entry == "verify_naive":
        ref.req_status.zero_()
        bad.req_status.zero_()
        ref.verify_naive(target, 0)
        bad.verify_naive(target, 0)
    else:
        bad.topk_tok.copy_(ref.topk_tok)
        bad.replay(draft, 1)
        ref.replay(draft, 1)
    torch.cuda.synchronize()
    a, b = ref.host(), bad.host()
    if entry == "replay":
        assert torch.equal(a["node_tok"][0], b["node_tok"][0])      # the clean request is untouched
        assert (b["node_tok"][5] == -1).all()                          # unusable n_nodes: nothing replayed
        return
    for k in ("n_acc", "acc_node", "acc_tok", "bonus", "req_status", "trace"):
        assert _same(a[k][0], b[k][0]), k
    flagged = [1, 2, 3, 5] if entry == "verify_naive" else [1, 2, 3, 4, 5]  # the Naive walk reads no depth
    for r in flagged:
        assert int(b["req_status"][r]) & tsb.REQ_BAD_TREE, (entry, r, int(b["req_status"][r]))
        assert int(b["n_acc"][r]) == -1 and int(b["bonus"][r]) == -1
        assert (b["acc_node"][r] == -1).all() and (b["acc_tok"][r] == -1).all()
    assert int((b["req_status"] & tsb.REQ_WALK_TIMEOUT).sum()) == 0


def test_out_of_range_tokens_are_flagged():
    rng = np.random.default_rng(9)
    draft = torch.from_numpy((rng.standard_normal((4, 4, 3000)) * 2).astype(np.float32)).cuda()
    target = torch.from_numpy((rng.standard_normal((4, 13, 3000)) * 2).astype(np.float32)).cuda()
    c = tsb.make_config(4, 4, 3000, 12, 3, 1.0, "f32", 4)
    ref = tsb.Round(c, "cuda", target_lse=True, trace=True)
    ref.plan(draft)
    ref.replay(draft, 0)
    bad = tsb.Round(c, "cuda", target_lse=True, trace=True)
    bad.load_tree(ref.tree)
    bad.draft_lse.copy_(ref.draft_lse)
    tok = ref.node_tok.clone()
    fc = ref.tree["first_child"][:, 0].long()
    tok[1, fc[1]] = 3000          # = V
    tok[2, fc[2]] = -7
    tok[3, fc[3] + 1] = 1 << 30
    bad.node_tok.copy_(tok)
    ref.req_status.zero_()
    bad.req_status.zero_()
    ref.verify(draft, target, 0)
    bad.verify(draft, target, 0)
    a, b = ref.host(), bad.host()
    for k in ("n_acc", "acc_node", "acc_tok", "bonus", "req_status"):
        assert _same(a[k][0], b[k][0]), k
    for r in (1, 2, 3):
        assert int(b["req_status"][r]) & tsb.REQ_BAD_TOKEN, r
        assert int(b["n_acc"][r]) == -1 and int(b["bonus"][r]) == -1
