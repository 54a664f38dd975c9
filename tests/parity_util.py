"""Helpers of the GPU parity tests: run the CPU oracle on the very bytes the
HIP path consumed and compare stage by stage.

Comparison rules (the numeric contract of the library):
  * integer / token / topology outputs: bit-exact, except decisions whose
    oracle margin is below NEAR_TIE (reported, then the rest of that request
    is not compared);
  * draft log-sum-exp (binary64): relative 1e-12; planning lp (binary32):
    bit-exact;
  * streamed target log-sum-exp: absolute 2e-6 (binary32 terms on the HIP
    side; the walk refines the normaliser of every node it tests in binary64);
  * acceptance ratios and residual masses: |g - o| <= 1e-5 |o| + 1e-7.
"""
import numpy as np
import torch

from oracle import planner, replay as oreplay, step as ostep
from oracle.rowstats import STATUS_NONFINITE
import paper_2609_33652_amd as tsb

NEAR_TIE = ostep.NEAR_TIE
# Streamed target normaliser: binary32 exp terms, whose argument rounding
# grows with |a - max| (about 2^-24 |a - max| relative per term), so the
# log-sum-exp is within a few 1e-7 for rows of entropy up to ~12 nats.
LSE_T_ATOL = 2e-6


def to_np(t):
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.detach().cpu().numpy()


def make_round(cfg_dict, seed, flags=0, trace=True):
    c = tsb.make_config(cfg_dict["R"], cfg_dict["D"], cfg_dict["V"], cfg_dict["B"], cfg_dict["K"],
                        cfg_dict["T"], cfg_dict["dtype"], seed, flags)
    return tsb.Round(c, "cuda", target_lse=True, trace=trace)


def tree_dict_np(h, r):
    n = int(h["n_nodes"][r])
    return dict(n_nodes=n, parent=h["parent"][r, :n].numpy().astype(np.int64),
                depth=h["depth"][r, :n].numpy().astype(np.int64), rank=h["rank"][r, :n].numpy().astype(np.int64),
                n_children=h["n_children"][r, :n].numpy().astype(np.int64),
                first_child=h["first_child"][r, :n].numpy().astype(np.int64),
                score=h["score"][r, :n].numpy(), plan_margin=float(h["plan_margin"][r]))


class Tally:
    def __init__(self):
        self.exact = 0
        self.flagged = 0
        self.notes = []

    def flag(self, what):
        self.flagged += 1
        self.notes.append(what)


def compare_plan(h, r, pl, tally, where=""):
    """GPU plan outputs of request r against oracle plan_request output. Returns True if equal."""
    o_tree = pl["tree"]
    if pl["status"] & STATUS_NONFINITE:
        assert int(h["req_status"][r]) & tsb.REQ_NONFINITE, where
        return False
    np.testing.assert_allclose(h["draft_lse"][r].numpy(), pl["lse64"], rtol=1e-12, atol=0, err_msg=where)
    lse32_equal = np.array_equal(h["draft_lse"][r].numpy().astype(np.float32), pl["lse32"])
    assert np.array_equal(h["topk_tok"][r].numpy(), pl["topk_tok"]), where
    if not lse32_equal:
        tally.flag("lse32 rounding differs " + where)
        return False
    assert np.array_equal(h["topk_lp"][r].numpy(), pl["topk_lp"]), where
    g = tree_dict_np(h, r)
    margin = o_tree["plan_margin"]
    if g["n_nodes"] != o_tree["n_nodes"] or not all(
            np.array_equal(g[k], o_tree[k]) for k in ("parent", "depth", "rank", "n_children", "first_child")):
        if 0 < margin < NEAR_TIE:
            tally.flag("plan near-tie %g %s" % (margin, where))
            return False
        raise AssertionError("topology differs %s (margin %g)" % (where, margin))
    assert np.array_equal(g["score"], o_tree["score"]), where
    if np.isfinite(margin):
        assert g["plan_margin"] == margin, where
    else:
        assert not np.isfinite(g["plan_margin"]), where
    tally.exact += 1
    return True


def compare_replay(gpu_tok, o_tok, margins, tally, where=""):
    if np.array_equal(gpu_tok, o_tok):
        tally.exact += 1
        return True
    if any(0 < m < NEAR_TIE for m in margins.values()):
        tally.flag("replay near-tie " + where)
        return False
    diff = np.nonzero(gpu_tok != o_tok)[0]
    raise AssertionError("node tokens differ at %s %s: gpu %s oracle %s"
                         % (where, diff[:8], gpu_tok[diff[:8]], o_tok[diff[:8]]))


def compare_verify(h, r, vr, tally, D, where=""):
    n_acc = int(h["n_acc"][r])
    got = (n_acc, list(h["acc_node"][r, :max(n_acc, 0)].numpy()), list(h["acc_tok"][r, :max(n_acc, 0)].numpy()),
           int(h["bonus"][r]))
    exp = (vr["n_acc"], list(vr["acc_node"]), list(vr["acc_tok"]), vr["bonus"])
    if vr["n_acc"] >= 0:
        # probabilities along the walk
        tr = h["trace"][r].numpy()
        nt = min(len(vr["tests"]), tr.shape[0])
        for i in range(nt):
            c, U, ratio, ok = vr["tests"][i]
            if int(tr[i, 0]) != c:
                break
            assert tr[i, 1] == U, where
            assert abs(tr[i, 2] - ratio) <= 1e-5 * abs(ratio) + 1e-7, (where, i, tr[i, 2], ratio)
        lt = h["target_lse"][r].numpy()[: len(vr["lse_t"])]
        tally.max_lse_err = max(getattr(tally, "max_lse_err", 0.0), float(np.abs(lt - vr["lse_t"]).max()))
        np.testing.assert_allclose(lt, vr["lse_t"], rtol=0, atol=LSE_T_ATOL, err_msg=where)
    if got == (exp[0], [int(x) for x in exp[1]], [int(x) for x in exp[2]], exp[3]):
        rest = [-1] * (D - max(n_acc, 0))
        assert list(h["acc_node"][r, max(n_acc, 0):].numpy()) == rest, where
        tally.exact += 1
        return True
    if any(0 < m[2] < NEAR_TIE for m in vr["margins"]):
        tally.flag("verify near-tie " + where)
        return False
    raise AssertionError("verification differs %s: gpu %s oracle %s" % (where, got, exp))


def oracle_replay_request(a_draft, tree, seed, step, r):
    return oreplay.replay(a_draft, tree, seed, step, r)


def budget_nodes(D, K):
    return planner.max_nodes(D, K)
