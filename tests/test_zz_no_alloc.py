"""tsb_step_noalloc (scratch in the library's per-device array) against
tsb_step (caller workspace), through the C ABI: two calls in a row, the
second on a smaller problem, both bit-identical to tsb_step on the same
inputs. The first call runs at the full batched serving shape (R = 16,
V = 151936, D = 16, B = 128, K = 10, bf16), the largest the fixed scratch
holds; the second reuses the array after it without any clearing by the
caller."""
import pytest
import torch

import workloads as W
import paper_2609_33652_amd as tsb

pytestmark = pytest.mark.gpu

KEYS = ("draft_lse", "topk_tok", "topk_lp", "parent", "depth", "rank", "n_children", "first_child", "score",
        "n_nodes", "plan_margin", "node_tok", "n_acc", "acc_node", "acc_tok", "bonus", "req_status", "target_lse",
        "trace")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    tsb.load()


def _inputs(cfg, device):
    base, sigma = W.base_rows(cfg, 0, device=device)
    draft = W.draft_from_base(cfg, base)
    c = tsb.make_config(cfg["R"], cfg["D"], cfg["V"], cfg["B"], cfg["K"], cfg["T"], cfg["dtype"],
                        W.replay_seed(cfg["id"]))
    rnd = tsb.Round(c, "cuda")
    rnd.plan(draft.cuda())
    dep = rnd.tree["depth"].long().clamp(min=0).to(base.device)
    target = W.target_from_base(cfg, base, sigma, dep)
    return c, draft.cuda(), target.cuda()


def _same(a, b):
    if a.dtype.is_floating_point:
        return torch.equal(a.nan_to_num(7.0), b.nan_to_num(7.0))
    return torch.equal(a, b)


def test_step_noalloc_equals_step_two_calls_second_smaller():
    cases = [(W.config(4), "cuda", 3), (W.config(2, R=3, V=32000, D=8, B=40, K=6, name="small3"), "cpu", 11)]
    for cfg, dev, step in cases:
        c, draft, target = _inputs(cfg, dev)
        assert tsb.workspace_bytes(c) <= tsb.NOALLOC_SCRATCH_BYTES
        a = tsb.Round(c, "cuda", target_lse=True, trace=True)
        b = tsb.Round(c, "cuda", target_lse=True, trace=True)
        a.step(draft, target, step)
        b.step_noalloc(draft, target, step)
        ha, hb = a.host(), b.host()
        for k in KEYS:
            assert _same(ha[k], hb[k]), (cfg["name"], k)
        assert int((hb["req_status"] & (tsb.REQ_WALK_TIMEOUT | tsb.REQ_NONFINITE)).sum()) == 0
        print("noalloc %s: n_acc %s" % (cfg["name"], hb["n_acc"].tolist()), flush=True)


def test_step_noalloc_rejects_oversized_configuration():
    cfg = W.config(5)
    c = tsb.make_config(cfg["R"], cfg["D"], cfg["V"], cfg["B"], cfg["K"], cfg["T"], cfg["dtype"], 1)
    rnd = tsb.Round(c, "cuda")
    draft = torch.zeros(cfg["R"], cfg["D"], cfg["V"], dtype=torch.bfloat16, device="cuda")
    target = torch.zeros(cfg["R"], cfg["B"] + 1, cfg["V"], dtype=torch.bfloat16, device="cuda")
    with pytest.raises(tsb.TsbError) as ei:
        rnd.step_noalloc(draft, target, 0)
    assert ei.value.status == 5
