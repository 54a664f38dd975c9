"""A round captured as a HIP graph (through torch.cuda.CUDAGraph) gives the
eager round's outputs on every replay.

The C ABI enqueues kernels only on the caller's stream, allocates nothing and
records no memset, so tsb_step can be captured. Each replay here is followed
by eager rounds of other step indices and synchronisations (which rewrite
every output buffer), and the replayed outputs are compared with an eager
round of the captured step index, bit for bit.
"""
import pytest
import torch

import workloads as W
import paper_2609_33652_amd as tsb

pytestmark = pytest.mark.gpu

KEYS = ("draft_lse", "topk_tok", "parent", "n_children", "first_child", "n_nodes", "node_tok", "n_acc",
        "acc_node", "acc_tok", "bonus", "req_status", "target_lse")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tsb.load()


def _inputs(cfg_id, target_lse=True):
    cfg = W.config(cfg_id)
    c = tsb.make_config(cfg["R"], cfg["D"], cfg["V"], cfg["B"], cfg["K"], cfg["T"], cfg["dtype"],
                        W.replay_seed(cfg_id))
    rnd = tsb.Round(c, "cuda", target_lse=target_lse)
    base, sigma = W.base_rows(cfg, 0, device="cuda")
    draft = W.draft_from_base(cfg, base)
    rnd.plan(draft)
    dep = rnd.tree["depth"].long().clamp(min=0)
    target = W.target_from_base(cfg, base, sigma, dep)
    return rnd, draft, target


def _snapshot(rnd):
    h = rnd.host()
    return {k: h[k].clone() for k in KEYS if h[k] is not None}


def _same(a, b):
    if a.dtype.is_floating_point:
        return torch.equal(a.nan_to_num(7.0), b.nan_to_num(7.0))
    return torch.equal(a, b)


@pytest.mark.parametrize("cfg_id,target_lse", [(1, True), (3, True), (4, True), (4, False)])
def test_captured_round_matches_eager(cfg_id, target_lse):
    """At the batched workload without the normaliser output the walk reads the rows of the nodes it
    enters (the scan's grid only clears the exchange slots); with it every row is streamed."""
    rnd, draft, target = _inputs(cfg_id, target_lse)
    step = 5
    rnd.step(draft, target, step)
    ref = _snapshot(rnd)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        rnd.step(draft, target, step)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        rnd.step(draft, target, step)
    for rep in range(3):
        # eager rounds of other steps rewrite every output between replays
        rnd.step(draft, target, 100 + rep)
        torch.cuda.synchronize()
        other = _snapshot(rnd)
        g.replay()
        torch.cuda.synchronize()
        got = _snapshot(rnd)
        for k in ref:
            assert _same(got[k], ref[k]), (cfg_id, rep, k)
        assert any(not _same(other[k], ref[k]) for k in ("node_tok", "n_acc", "bonus")), (cfg_id, rep)
    del g
