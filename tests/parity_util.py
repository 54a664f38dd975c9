"""GPU-versus-oracle parity harness: runs the CPU oracle on the very bytes
the HIP path consumed (in a process pool for the large workloads) and
compares stage by stage, decision by decision.

Comparison rules (the numeric contract of the library). A difference is
excused only at the one decision that produced it, and only when that
decision's own oracle margin is below NEAR_TIE (1e-5 in the decision's
units); it is then counted as flagged. Any other difference fails the test.

  plan    draft log-sum-exp (binary64) within 1e-12 relative; its canonical
          binary32 rounding equal, except a row whose oracle value lies within
          1e-12 relative of a binary32 rounding boundary (flagged); candidate
          tokens and lp bit-exact; topology, scores and plan_margin bit-exact,
          except a plan whose oracle margin is below NEAR_TIE (flagged).
  replay  parent by parent: the m tokens of a parent bit-exact, except a
          parent whose own oracle margin (smallest gap among its m + 1
          largest keys) is below NEAR_TIE (flagged).
  verify  test by test along the walk: child and uniform bit-exact, ratio and
          residual mass within |g - o| <= 1e-5 |o| + 1e-7; the first test whose
          accept/reject outcome differs is excused only if its own oracle
          margin |U - ratio| is below NEAR_TIE (flagged; the rest of that walk
          is not compared); otherwise the accepted path and n_acc are exact
          and the bonus is exact unless its own oracle margin (gap between
          the two largest bonus keys) is below NEAR_TIE (flagged).
  target  streamed log-sum-exp of every node row within 2e-6 absolute.
"""
import atexit
import multiprocessing as mp
import os
import shutil
import tempfile

import numpy as np
import torch

import oracle_worker
from oracle import planner, step as ostep
from oracle.rowstats import STATUS_BUDGET_SHORT, STATUS_DEGENERATE_RESIDUAL, STATUS_NONFINITE
import paper_2609_33652_amd as tsb
from tally import Tally

NEAR_TIE = ostep.NEAR_TIE
# Streamed target normaliser: binary32 exp terms, whose argument rounding
# grows with |a - max| (about 2^-24 |a - max| relative per term), so the
# log-sum-exp is within a few 1e-7 for rows of entropy up to ~12 nats.
LSE_T_ATOL = 2e-6
PROB_RTOL, PROB_ATOL = 1e-5, 1e-7


def to_np(t):
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.detach().cpu().numpy()


def make_round(cfg_dict, seed, flags=0, trace=True, target_lse=True):
    c = tsb.make_config(cfg_dict["R"], cfg_dict["D"], cfg_dict["V"], cfg_dict["B"], cfg_dict["K"],
                        cfg_dict["T"], cfg_dict["dtype"], seed, flags)
    return tsb.Round(c, "cuda", target_lse=target_lse, trace=trace)


def tree_dict_np(h, r):
    n = int(h["n_nodes"][r])
    return dict(n_nodes=n, parent=h["parent"][r, :n].numpy().astype(np.int64),
                depth=h["depth"][r, :n].numpy().astype(np.int64), rank=h["rank"][r, :n].numpy().astype(np.int64),
                n_children=h["n_children"][r, :n].numpy().astype(np.int64),
                first_child=h["first_child"][r, :n].numpy().astype(np.int64),
                score=h["score"][r, :n].numpy(), plan_margin=float(h["plan_margin"][r]))


def _close(g, o):
    return g == o or abs(g - o) <= PROB_RTOL * abs(o) + PROB_ATOL


def near_f32_boundary(x, rel=1e-12):
    """True if binary64 x lies within rel |x| of a point where its binary32 rounding changes."""
    f = np.float32(x)
    if not np.isfinite(f):
        return False
    nb = np.nextafter(f, np.float32(np.inf) if float(f) < x else np.float32(-np.inf))
    mid = (float(f) + float(nb)) / 2.0
    return abs(x - mid) <= rel * abs(x)


# ---------------------------------------------------------------- stages
def compare_plan(h, r, pl, tally, where=""):
    """GPU plan outputs of request r against oracle plan_request output. Returns 'exact' or 'flagged'."""
    o_tree = pl["tree"]
    if pl["status"] & STATUS_NONFINITE:
        assert int(h["req_status"][r]) & tsb.REQ_NONFINITE, where
        tally.ok("plan")
        return "exact"
    g64 = h["draft_lse"][r].numpy()
    np.testing.assert_allclose(g64, pl["lse64"], rtol=1e-12, atol=0, err_msg=where)
    assert np.array_equal(h["topk_tok"][r].numpy(), pl["topk_tok"]), where
    g32 = g64.astype(np.float32)
    diff = np.nonzero(g32 != pl["lse32"])[0]
    for d in diff:
        if not near_f32_boundary(float(pl["lse64"][d])):
            raise AssertionError("binary32 normaliser differs at row %d away from a rounding boundary %s "
                                 "(gpu %r oracle %r)" % (d, where, g64[d], pl["lse64"][d]))
    if diff.size:
        tally.flag("plan", "lse32 at a rounding boundary " + where)
        return "flagged"
    assert np.array_equal(h["topk_lp"][r].numpy(), pl["topk_lp"]), where
    g = tree_dict_np(h, r)
    margin = o_tree["plan_margin"]
    if g["n_nodes"] != o_tree["n_nodes"] or not all(
            np.array_equal(g[k], o_tree[k]) for k in ("parent", "depth", "rank", "n_children", "first_child")):
        if 0 < margin < NEAR_TIE:
            tally.flag("plan", "plan near-tie %g %s" % (margin, where))
            return "flagged"
        raise AssertionError("topology differs %s (margin %g)" % (where, margin))
    assert np.array_equal(g["score"], o_tree["score"]), where
    if np.isfinite(margin):
        assert g["plan_margin"] == margin, where
    else:
        assert not np.isfinite(g["plan_margin"]), where
    tally.ok("plan")
    return "exact"


def compare_replay(gpu_tok, o_tok, margins, tree, tally, where=""):
    """Node tokens parent by parent (tree in oracle format, margins: parent -> margin)."""
    out = "exact"
    for u in range(tree["n_nodes"]):
        m = int(tree["n_children"][u])
        if m == 0:
            continue
        fc = int(tree["first_child"][u])
        g, o = gpu_tok[fc:fc + m], o_tok[fc:fc + m]
        if np.array_equal(g, o):
            tally.ok("replay")
            continue
        mg = margins[u]
        if 0 < mg < NEAR_TIE:
            tally.flag("replay", "replay near-tie %.2e at parent %d %s" % (mg, u, where))
            out = "flagged"
            continue
        raise AssertionError("node tokens of parent %d differ %s: gpu %s oracle %s (margin %g)"
                             % (u, where, g, o, mg))
    assert gpu_tok[0] == -1, where
    return out


def compare_verify(h, r, vr, tree, tally, D, where=""):
    """The walk of request r decision by decision (trace), then its outputs."""
    n_acc = int(h["n_acc"][r])
    st = int(h["req_status"][r])
    if vr["n_acc"] < 0:
        assert n_acc == -1 and st & tsb.REQ_NONFINITE and int(h["bonus"][r]) == -1, where
        tally.ok("verify")
        return "exact"
    tr = h["trace"][r].numpy()
    tests, zs = vr["tests"], vr["residual_Z"]
    parent = tree["parent"]
    zi, prod, cur = 0, 1.0, None
    nt = min(len(tests), tr.shape[0])
    for i in range(nt):
        c, U, ratio, ok = tests[i]
        gc, gU, gr, gz = tr[i]
        if int(gc) != c:
            raise AssertionError("walk tests child %d where the oracle tests %d %s (test %d)" % (int(gc), c, where, i))
        assert gU == U, (where, i, gU, U)
        assert _close(gr, ratio), (where, i, "ratio", gr, ratio)
        g_ok = gU < gr
        if g_ok != ok:
            mg = abs(U - ratio)
            if 0 < mg < NEAR_TIE:
                tally.flag("verify", "accept near-tie %.2e at test %d %s" % (mg, i, where))
                return "flagged"
            raise AssertionError("acceptance of child %d differs %s: gpu U %r ratio %r, oracle ratio %r"
                                 % (c, where, gU, gr, ratio))
        u = int(parent[c])
        if u != cur:
            cur, prod = u, 1.0
        if not ok:
            prod *= zs[zi]
            zi += 1
            if prod > 0.0:
                assert gz >= 0.0 and _close(gz, prod), (where, i, "residual mass", gz, prod)
    if len(tests) <= tr.shape[0]:
        assert int((tr[:, 0] >= 0).sum()) == len(tests), (where, "trace length")
    exp_path = ([int(x) for x in vr["acc_node"]], [int(x) for x in vr["acc_tok"]])
    got_path = (list(h["acc_node"][r, :max(n_acc, 0)].numpy()), list(h["acc_tok"][r, :max(n_acc, 0)].numpy()))
    if n_acc != vr["n_acc"] or got_path != exp_path:
        raise AssertionError("accepted path differs with every test agreeing %s: gpu %s oracle %s"
                             % (where, (n_acc, got_path), (vr["n_acc"], exp_path)))
    assert list(h["acc_node"][r, n_acc:].numpy()) == [-1] * (D - n_acc), where
    assert bool(st & tsb.REQ_DEGENERATE_RESIDUAL) == bool(vr["status"] & STATUS_DEGENERATE_RESIDUAL), where
    lt = h["target_lse"][r].numpy()[: len(vr["lse_t"])]
    err = float(np.abs(lt - vr["lse_t"]).max())
    tally.max_lse_err = max(tally.max_lse_err, err)
    np.testing.assert_allclose(lt, vr["lse_t"], rtol=0, atol=LSE_T_ATOL, err_msg=where)
    if int(h["bonus"][r]) != vr["bonus"]:
        mg = [m for m in vr["margins"] if m[0] == "bonus"][-1][2]
        if 0 < mg < NEAR_TIE:
            tally.flag("verify", "bonus near-tie %.2e %s" % (mg, where))
            return "flagged"
        raise AssertionError("bonus differs %s: gpu %d oracle %d (margin %g)" % (where, int(h["bonus"][r]),
                                                                                  vr["bonus"], mg))
    tally.ok("verify")
    return "exact"


def compare_naive(h, r, vr, tally, D, where=""):
    """Target-sample matching walk of request r. The GPU reports its path and bonus; the first index where
    the paths part (or the bonus, when the paths agree) is the first differing draw, excused only if that
    draw's own oracle margin is below NEAR_TIE."""
    n_acc = int(h["n_acc"][r])
    st = int(h["req_status"][r])
    if vr["n_acc"] < 0:
        assert n_acc == -1 and st & tsb.REQ_NONFINITE and int(h["bonus"][r]) == -1, where
        tally.ok("verify")
        return "exact"
    assert not st & (tsb.REQ_NONFINITE | tsb.REQ_WALK_TIMEOUT | tsb.REQ_BAD_TREE), where
    g_node = [int(x) for x in h["acc_node"][r, :max(n_acc, 0)]]
    g_tok = [int(x) for x in h["acc_tok"][r, :max(n_acc, 0)]]
    o_node, o_tok = [int(x) for x in vr["acc_node"]], [int(x) for x in vr["acc_tok"]]
    assert [int(x) for x in h["acc_node"][r, max(n_acc, 0):]] == [-1] * (D - max(n_acc, 0)), where
    i = 0
    while i < min(len(g_node), len(o_node)) and g_node[i] == o_node[i] and g_tok[i] == o_tok[i]:
        i += 1
    same_path = i == len(g_node) == len(o_node)
    if same_path and int(h["bonus"][r]) == int(vr["bonus"]):
        tally.ok("verify")
        return "exact"
    mg = vr["margins"][i][1]  # the draw at the i-th visited node (the terminal one when the paths agree)
    if 0 < mg < NEAR_TIE:
        tally.flag("verify", "naive draw near-tie %.2e at visited node %d %s" % (mg, i, where))
        return "flagged"
    raise AssertionError("naive verification differs %s at visited node %d: gpu %s oracle %s (margin %g)"
                         % (where, i, (n_acc, g_node, g_tok, int(h["bonus"][r])),
                            (vr["n_acc"], o_node, o_tok, vr["bonus"]), mg))


def compare_request_naive(h, r, res, tally, D, where):
    """Plan, First tokens and target-sample matching of one request-step."""
    compare_plan(h, r, res["plan"], tally, where)
    tally.request_steps += 1
    if res["first_tok"] is None:
        assert int(h["req_status"][r]) & tsb.REQ_NONFINITE and int(h["n_acc"][r]) == -1, where
        return
    n = int(h["n_nodes"][r])
    if n == res["plan"]["tree"]["n_nodes"]:
        g = h["node_tok"][r, :n].numpy().astype(np.int64)
        if np.array_equal(g, res["first_tok"]):
            tally.ok("replay")
        else:
            raise AssertionError("First tokens differ %s" % where)
    if res["naive"] is not None:
        compare_naive(h, r, res["naive"], tally, D, where)


def compare_traversal(h, r, vr, tree, tally, D, where=""):
    """The traversal of request r test by test (trace rows: tested node, U, alpha, T after its rejection),
    then its outputs. The first test whose outcome differs is excused only at its own oracle margin."""
    n_acc = int(h["n_acc"][r])
    st = int(h["req_status"][r])
    if vr["n_acc"] < 0:
        assert n_acc == -1 and st & tsb.REQ_NONFINITE and int(h["bonus"][r]) == -1, where
        tally.ok("verify")
        return "exact"
    tr = h["trace"][r].numpy()
    tests, Ts = vr["tests"], vr["residual_T"]
    zi = 0
    for i in range(min(len(tests), tr.shape[0])):
        u, U, alpha, ok = tests[i]
        gu, gU, ga, gT = tr[i]
        if int(gu) != u:
            raise AssertionError("traversal tests node %d where the oracle tests %d %s (test %d)"
                                 % (int(gu), u, where, i))
        assert gU == U, (where, i, gU, U)
        assert _close(ga, alpha), (where, i, "alpha", ga, alpha)
        g_ok = gU < ga
        if g_ok != ok:
            mg = abs(U - alpha)
            if 0 < mg < NEAR_TIE:
                tally.flag("verify", "traversal near-tie %.2e at test %d %s" % (mg, i, where))
                return "flagged"
            raise AssertionError("acceptance of node %d differs %s: gpu U %r alpha %r, oracle alpha %r"
                                 % (u, where, gU, ga, alpha))
        if not ok:
            if zi < len(Ts):
                assert _close(gT, Ts[zi]), (where, i, "residual mass", gT, Ts[zi])
            zi += 1
    if len(tests) <= tr.shape[0]:
        assert int((tr[:, 0] >= 0).sum()) == len(tests), (where, "trace length")
    exp_path = ([int(x) for x in vr["acc_node"]], [int(x) for x in vr["acc_tok"]])
    got_path = (list(h["acc_node"][r, :max(n_acc, 0)].numpy()), list(h["acc_tok"][r, :max(n_acc, 0)].numpy()))
    if n_acc != vr["n_acc"] or got_path != exp_path:
        raise AssertionError("accepted path differs with every test agreeing %s: gpu %s oracle %s"
                             % (where, (n_acc, got_path), (vr["n_acc"], exp_path)))
    assert list(h["acc_node"][r, n_acc:].numpy()) == [-1] * (D - n_acc), where
    assert bool(st & tsb.REQ_DEGENERATE_RESIDUAL) == bool(vr["status"] & STATUS_DEGENERATE_RESIDUAL), where
    assert not st & (tsb.REQ_WALK_TIMEOUT | tsb.REQ_BAD_TREE | tsb.REQ_BAD_TOKEN), where
    lt = h["target_lse"][r].numpy()[: len(vr["lse_t"])]
    tally.max_lse_err = max(tally.max_lse_err, float(np.abs(lt - vr["lse_t"]).max()))
    np.testing.assert_allclose(lt, vr["lse_t"], rtol=0, atol=LSE_T_ATOL, err_msg=where)
    if int(h["bonus"][r]) != vr["bonus"]:
        mg = [m for m in vr["margins"] if m[0] == "bonus"][-1][2]
        if 0 < mg < NEAR_TIE:
            tally.flag("verify", "traversal bonus near-tie %.2e %s" % (mg, where))
            return "flagged"
        raise AssertionError("bonus differs %s: gpu %d oracle %d (margin %g)" % (where, int(h["bonus"][r]),
                                                                                  vr["bonus"], mg))
    tally.ok("verify")
    return "exact"


def compare_request_traversal(h, r, res, tally, D, where):
    """Plan, replay and traversal verification of one request-step."""
    compare_plan(h, r, res["plan"], tally, where)
    tally.request_steps += 1
    if res["replay"] is None:
        assert int(h["req_status"][r]) & tsb.REQ_NONFINITE or int(h["n_nodes"][r]) == 1, where
        return
    tree = tree_dict_np(h, r)
    n = tree["n_nodes"]
    o_tok, mg = res["replay"]
    compare_replay(h["node_tok"][r, :n].numpy().astype(np.int64), o_tok, mg, tree, tally, where)
    if res["verify"] is not None:
        compare_traversal(h, r, res["verify"], tree, tally, D, where)


def compare_request(h, r, res, tally, D, where):
    """All three stages of one request-step (res: oracle_worker.request_step output)."""
    compare_plan(h, r, res["plan"], tally, where)
    tally.request_steps += 1
    if res["replay"] is None:
        assert int(h["req_status"][r]) & tsb.REQ_NONFINITE or int(h["n_nodes"][r]) == 1, where
        return
    tree = tree_dict_np(h, r)
    n = tree["n_nodes"]
    o_tok, mg = res["replay"]
    compare_replay(h["node_tok"][r, :n].numpy().astype(np.int64), o_tok, mg, tree, tally, where)
    if res["verify"] is not None:
        compare_verify(h, r, res["verify"], tree, tally, D, where)


# ---------------------------------------------------------------- oracle pool
def worker_count():
    """Processes for the oracle: the CPUs this process may use, at most 16."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


class OraclePool:
    """A spawn-context process pool running oracle_worker.run, with the logits shared through files."""

    def __init__(self):
        self.n = worker_count()
        self.pool = mp.get_context("spawn").Pool(self.n)
        base = "/dev/shm" if os.path.isdir("/dev/shm") and os.access("/dev/shm", os.W_OK) else None
        self.dir = tempfile.mkdtemp(prefix="tsb_parity_", dir=base)
        atexit.register(self.close)

    def put(self, name, t):
        """Write a logit tensor (host or device) to a shared file; returns its spec."""
        t = t.detach().cpu().contiguous()
        path = os.path.join(self.dir, name)
        if t.dtype == torch.bfloat16:
            t.view(torch.int16).numpy().tofile(path)
            return (path, tuple(t.shape), "bf16")
        t.float().numpy().tofile(path)
        return (path, tuple(t.shape), "f32")

    def drop(self, *specs):
        for s in specs:
            if s is not None and os.path.exists(s[0]):
                os.remove(s[0])

    def close(self):
        if self.pool is not None:
            self.pool.terminate()
            self.pool.join()
            self.pool = None
        shutil.rmtree(self.dir, ignore_errors=True)


def compare_request_pool(h, r, res, tally, D, where):
    """Pools, first pass over per-node candidate lists, replay and the pool walk of one request-step."""
    tally.request_steps += 1
    st = int(h["req_status"][r])
    if res["status"] & STATUS_NONFINITE:
        assert st & tsb.REQ_NONFINITE and int(h["n_nodes"][r]) == 1 and int(h["n_acc"][r]) == -1, where
        tally.ok("plan")
        return
    assert np.array_equal(h["pool_tok"][r].numpy().astype(np.int64), res["pool"]), where
    tree = res["tree"]
    g = tree_dict_np(h, r)
    margin = tree["plan_margin"]
    same = g["n_nodes"] == tree["n_nodes"] and all(
        np.array_equal(g[k], tree[k]) for k in ("parent", "depth", "rank", "n_children", "first_child"))
    if same:
        assert np.array_equal(g["score"], tree["score"]), where
        assert (g["plan_margin"] == margin) if np.isfinite(margin) else not np.isfinite(g["plan_margin"]), where
        n = tree["n_nodes"]
        assert np.array_equal(h["plan_tok"][r, :n].numpy().astype(np.int64), res["plan_tok"]), where
        assert bool(st & tsb.REQ_BUDGET_SHORT) == bool(res["status"] & STATUS_BUDGET_SHORT), where
        tally.ok("plan")
    elif 0 < margin < NEAR_TIE:
        tally.flag("plan", "pool plan near-tie %g %s" % (margin, where))
    else:
        raise AssertionError("pool topology differs %s (margin %g)" % (where, margin))
    if res["replay"] is None:
        return
    n = g["n_nodes"]
    o_tok, mg = res["replay"]
    compare_replay(h["node_tok"][r, :n].numpy().astype(np.int64), o_tok, mg, g, tally, where)
    if res["verify"] is not None:
        assert not st & tsb.REQ_BAD_TOKEN, where
        compare_verify(h, r, res["verify"], g, tally, D, where)


COMPARE = {"rrs": compare_request, "naive": compare_request_naive, "pool": compare_request_pool,
           "traversal": compare_request_traversal}


def run_rounds(pool, cfg, seed, steps, kind, gpu_round, step0=0, sets=4, gen_device="cpu", name="", check=None,
               trace=True, P=None):
    """Parity of every request for rounds step0 .. step0 + steps - 1 of a workload.

    Per round: draft rows from the seeded generator; the HIP plan (its depths
    key the target rows); gpu_round(rnd, draft, target, s) runs the remaining
    HIP stages; check(h, draft, target, s), if given, compares a fused entry
    point with the staged one. The oracle tasks of round s (kind "rrs" or
    "naive") run in the pool while round s + 1 is prepared on the GPU, and
    every request is compared stage by stage."""
    import collections

    import workloads as W
    R, D, B, K, T = cfg["R"], cfg["D"], cfg["B"], cfg["K"], cfg["T"]
    if P is None:
        rnd = make_round(cfg, seed, trace=trace)
    else:
        c = tsb.make_config(R, D, cfg["V"], B, K, T, cfg["dtype"], seed)
        rnd = tsb.Round(c, "cuda", target_lse=True, trace=trace, pool=P)
    label = "" if kind == "rrs" else " (%s%s)" % (kind, "" if P is None else " P=%d" % P)
    tally = Tally("%s%s steps %d..%d" % (name, label, step0, step0 + steps - 1))
    compare = COMPARE[kind]
    # rounds in flight: enough to keep every worker busy when a round has few
    # requests, within a budget for the shared input files
    max_pending = max(1, min(2 * pool.n, (8 << 30) // max(1, W.bytes_per_step(cfg))))
    pending = collections.deque()

    def finish(p):
        h, job, specs = p
        for r, step, res in job.get():
            compare(h, r, res, tally, D, "%s step %d req %d" % (name, step, r))
        pool.drop(*specs)
        tally.steps += 1

    for s in range(step0, step0 + steps):
        base, sigma = W.base_rows(cfg, set_idx=s % sets, device=gen_device)
        draft = W.draft_from_base(cfg, base)
        draft_g = draft.cuda().contiguous()
        trans = trans_g = None
        if P is None:
            rnd.plan(draft_g)
        else:
            trans = W.transitions(cfg, P, set_idx=s % sets, device=gen_device)
            trans_g = trans.cuda().contiguous()
            rnd.pool_plan(draft_g, trans_g)
        dep = rnd.tree["depth"].long().clamp(min=0)
        target = W.target_from_base(cfg, base, sigma, dep.to(base.device), set_idx=s % sets)
        del base
        target_g = target.cuda().contiguous()
        if P is None:
            gpu_round(rnd, draft_g, target_g, s)
        else:
            gpu_round(rnd, draft_g, target_g, s, trans_g)
        h = rnd.host()
        if check is not None:
            check(h, draft_g, target_g, s) if P is None else check(h, draft_g, target_g, s, trans_g)
        specs = (pool.put("%s_d%d" % (name, s), draft), pool.put("%s_t%d" % (name, s), target))
        extra = ()
        if P is not None:
            specs = specs + (pool.put("%s_c%d" % (name, s), trans),)
            extra = (specs[2], P)
        del draft, target, draft_g, target_g, trans, trans_g
        tasks = [(kind, specs[0], specs[1], T, K, B, seed, s, r, tree_dict_np(h, r),
                  h["node_tok"][r, :int(h["n_nodes"][r])].numpy().astype(np.int64)) + extra for r in range(R)]
        pending.append((h, pool.pool.map_async(oracle_worker.run, tasks, chunksize=1), specs))
        while len(pending) > max_pending:
            finish(pending.popleft())
        if s % 20 == 0 or R > 1:
            print("case %s (%s): round %d prepared" % (name, kind, s), flush=True)
    while pending:
        finish(pending.popleft())
    print(tally.line(), flush=True)
    return tally


def check_tally(t, steps, R, max_flagged=1):
    """Every request of every round was compared; at most max_flagged near-ties were excused."""
    assert t.steps == steps and t.request_steps == steps * R, (t.steps, t.request_steps)
    assert t.flagged <= max_flagged, t.notes
    assert t.exact["plan"] + t.flagged_by["plan"] == steps * R


def budget_nodes(D, K):
    return planner.max_nodes(D, K)
