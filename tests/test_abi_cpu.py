"""C-ABI checks that need no GPU: the library loads, exports every entry
point declared in include/tsubame.h, and rejects invalid arguments on the
host before anything is enqueued (no HIP call is made by these cases)."""
import ctypes
import os
import re

import pytest

import paper_2609_33652_amd as tsb
from paper_2609_33652_amd import TsbConfig, TsbTree, TsbVerdict

HERE = os.path.dirname(os.path.abspath(__file__))
HEADER = os.path.join(HERE, "..", "include", "tsubame.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(tsb.LIB_PATH):
        from paper_2609_33652_amd import build
        build.build()
    return tsb.load()


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tsb_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert set(names) == set(tsb.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n
    assert lib.tsb_version() == 201


def _cfg(**kw):
    base = dict(R=2, D=4, V=1000, B=10, K=4, temperature=1.0, dtype="bf16", seed=1)
    base.update(kw)
    return tsb.make_config(**base)


FAKE = ctypes.c_void_p(0x100000)  # never dereferenced: validation fails first


def _tree():
    return TsbTree(**{n: 0x100000 for n, _ in TsbTree._fields_})


def _verdict():
    return TsbVerdict(n_acc=0x100000, acc_node=0x100000, acc_tok=0x100000, bonus=0x100000,
                      req_status=0x100000, target_lse=None, trace=None)


@pytest.mark.parametrize("kw,code", [
    (dict(R=0), 2), (dict(D=0), 2), (dict(D=65), 2), (dict(K=0), 2), (dict(K=33), 2),
    (dict(V=3, K=4), 2), (dict(B=-1), 2), (dict(B=1024), 2), (dict(dtype=7), 3),
    (dict(temperature=0.0), 4), (dict(temperature=float("nan")), 4), (dict(temperature=-1.0), 4),
    (dict(temperature=float("inf")), 4),
])
def test_invalid_config_rejected(lib, kw, code):
    cfg = _cfg(**kw)
    assert lib.tsb_workspace_bytes(ctypes.byref(cfg)) == 0
    t = _tree()
    st = lib.tsb_plan(ctypes.byref(cfg), FAKE, FAKE, FAKE, FAKE, ctypes.byref(t), FAKE, FAKE, 1 << 30, None)
    assert st == code
    assert lib.tsb_last_error().decode()
    v = _verdict()
    assert lib.tsb_step(ctypes.byref(cfg), FAKE, FAKE, 0, FAKE, FAKE, FAKE, ctypes.byref(t), FAKE,
                        ctypes.byref(v), FAKE, 1 << 30, None) == code


def test_null_pointers_rejected(lib):
    cfg = _cfg()
    t = _tree()
    v = _verdict()
    assert lib.tsb_plan(None, FAKE, FAKE, FAKE, FAKE, ctypes.byref(t), FAKE, FAKE, 1 << 30, None) == 1
    assert lib.tsb_plan(ctypes.byref(cfg), None, FAKE, FAKE, FAKE, ctypes.byref(t), FAKE, FAKE, 1 << 30, None) == 1
    assert lib.tsb_replay(ctypes.byref(cfg), FAKE, None, ctypes.byref(t), 0, FAKE, FAKE, 1 << 30, None) == 1
    bad_tree = _tree()
    bad_tree.score = None
    assert lib.tsb_replay(ctypes.byref(cfg), FAKE, FAKE, ctypes.byref(bad_tree), 0, FAKE, FAKE, 1 << 30, None) == 1
    bad_v = _verdict()
    bad_v.bonus = None
    assert lib.tsb_verify(ctypes.byref(cfg), FAKE, FAKE, FAKE, ctypes.byref(t), FAKE, 0, ctypes.byref(bad_v),
                          FAKE, 1 << 30, None) == 1
    assert lib.tsb_verify(ctypes.byref(cfg), FAKE, FAKE, FAKE, ctypes.byref(t), FAKE, 0, ctypes.byref(v),
                          None, 1 << 30, None) == 1


def test_workspace_checks(lib):
    cfg = _cfg()
    need = lib.tsb_workspace_bytes(ctypes.byref(cfg))
    assert need >= 256 and need % 256 == 0
    t = _tree()
    # too small
    assert lib.tsb_plan(ctypes.byref(cfg), FAKE, FAKE, FAKE, FAKE, ctypes.byref(t), FAKE, FAKE, need - 1,
                        None) == 5
    # misaligned
    assert lib.tsb_plan(ctypes.byref(cfg), FAKE, FAKE, FAKE, FAKE, ctypes.byref(t), FAKE,
                        ctypes.c_void_p(0x100010), need, None) == 5
    # grows with the problem
    big = _cfg(R=64, D=32, V=151936, B=256, K=16)
    assert lib.tsb_workspace_bytes(ctypes.byref(big)) > need


def test_status_strings(lib):
    for code in range(0, 8):
        assert lib.tsb_status_string(code).decode()
    assert lib.tsb_status_string(99).decode() == "unknown status"


def test_first_naive_entry_points_validate(lib):
    cfg = _cfg()
    need = lib.tsb_workspace_bytes(ctypes.byref(cfg))
    t = _tree()
    v = _verdict()
    bad = _cfg(K=0)
    assert lib.tsb_first_tokens(ctypes.byref(bad), FAKE, ctypes.byref(t), FAKE, None) == 2
    assert lib.tsb_first_tokens(ctypes.byref(cfg), None, ctypes.byref(t), FAKE, None) == 1
    assert lib.tsb_first_tokens(ctypes.byref(cfg), FAKE, ctypes.byref(t), None, None) == 1
    assert lib.tsb_verify_naive(ctypes.byref(_cfg(temperature=0.0)), FAKE, ctypes.byref(t), FAKE, 0,
                                ctypes.byref(v), FAKE, need, None) == 4
    assert lib.tsb_verify_naive(ctypes.byref(cfg), None, ctypes.byref(t), FAKE, 0, ctypes.byref(v), FAKE, need,
                                None) == 1
    bad_v = _verdict()
    bad_v.req_status = None
    assert lib.tsb_verify_naive(ctypes.byref(cfg), FAKE, ctypes.byref(t), FAKE, 0, ctypes.byref(bad_v), FAKE,
                                need, None) == 1
    assert lib.tsb_verify_naive(ctypes.byref(cfg), FAKE, ctypes.byref(t), FAKE, 0, ctypes.byref(v), FAKE,
                                need - 1, None) == 5
    assert lib.tsb_step_first(ctypes.byref(cfg), FAKE, None, 0, FAKE, FAKE, FAKE, ctypes.byref(t), FAKE,
                              ctypes.byref(v), FAKE, need, None) == 1
    assert lib.tsb_step_first(ctypes.byref(_cfg(dtype=9)), FAKE, FAKE, 0, FAKE, FAKE, FAKE, ctypes.byref(t),
                              FAKE, ctypes.byref(v), FAKE, need, None) == 3


def test_plan_ep_validates_frontier_and_size(lib):
    cfg = _cfg()
    need = lib.tsb_workspace_bytes(ctypes.byref(cfg))
    t = _tree()
    for w in (0, -1, 65):
        assert lib.tsb_plan_ep(ctypes.byref(cfg), w, FAKE, FAKE, FAKE, FAKE, ctypes.byref(t), FAKE, FAKE, need,
                               None) == 2
    big = _cfg(K=32, D=64, B=100)
    nb = lib.tsb_workspace_bytes(ctypes.byref(big))
    assert lib.tsb_plan_ep(ctypes.byref(big), 64, FAKE, FAKE, FAKE, FAKE, ctypes.byref(t), FAKE, FAKE, nb,
                           None) == 2
    assert "generates more nodes" in lib.tsb_last_error().decode()
    assert lib.tsb_plan_ep(ctypes.byref(cfg), 4, None, FAKE, FAKE, FAKE, ctypes.byref(t), FAKE, FAKE, need,
                           None) == 1
    assert lib.tsb_plan_ep(ctypes.byref(cfg), 4, FAKE, FAKE, FAKE, FAKE, ctypes.byref(t), FAKE, FAKE, need - 1,
                           None) == 5


def test_pool_entry_points_validate(lib):
    cfg = _cfg()
    need = lib.tsb_pool_workspace_bytes(ctypes.byref(cfg), 16)
    assert need >= 256 and need % 256 == 0
    assert lib.tsb_pool_workspace_bytes(ctypes.byref(cfg), 64) > need
    # pool size outside [K, min(64, V)]
    for P in (3, 65, 0):
        assert lib.tsb_pool_workspace_bytes(ctypes.byref(cfg), P) == 0
    assert lib.tsb_pool_workspace_bytes(ctypes.byref(_cfg(V=20, K=4)), 21) == 0
    t = _tree()
    v = _verdict()
    for P in (3, 65):
        assert lib.tsb_pool_plan(ctypes.byref(cfg), P, FAKE, FAKE, FAKE, ctypes.byref(t), None, FAKE, FAKE,
                                 need, None) == 2
    # transition table required with D > 1, optional with D = 1
    assert lib.tsb_pool_plan(ctypes.byref(cfg), 16, FAKE, None, FAKE, ctypes.byref(t), None, FAKE, FAKE, need,
                             None) == 1
    assert lib.tsb_pool_replay(ctypes.byref(cfg), 16, FAKE, None, FAKE, ctypes.byref(t), 0, FAKE, None) == 1
    assert lib.tsb_pool_plan(ctypes.byref(cfg), 16, FAKE, FAKE, None, ctypes.byref(t), None, FAKE, FAKE, need,
                             None) == 1
    assert lib.tsb_pool_plan(ctypes.byref(cfg), 16, FAKE, FAKE, FAKE, ctypes.byref(t), None, FAKE, FAKE,
                             need - 1, None) == 5
    assert lib.tsb_pool_verify(ctypes.byref(cfg), 16, FAKE, FAKE, FAKE, None, ctypes.byref(t), FAKE, 0,
                               ctypes.byref(v), FAKE, need, None) == 1
    assert lib.tsb_pool_verify(ctypes.byref(_cfg(temperature=0.0)), 16, FAKE, FAKE, FAKE, FAKE, ctypes.byref(t),
                               FAKE, 0, ctypes.byref(v), FAKE, need, None) == 4
    assert lib.tsb_pool_step(ctypes.byref(cfg), 16, FAKE, FAKE, FAKE, 0, FAKE, ctypes.byref(t), FAKE,
                             ctypes.byref(v), FAKE, need - 256, None) == 5
    assert lib.tsb_pool_step(ctypes.byref(_cfg(dtype=5)), 16, FAKE, FAKE, FAKE, 0, FAKE, ctypes.byref(t), FAKE,
                             ctypes.byref(v), FAKE, need, None) == 3


def test_step_noalloc_validates_before_any_device_call(lib):
    """tsb_step_noalloc rejects a configuration whose scratch exceeds the library's fixed per-device array, and
    invalid arguments, on the host (no HIP call is made, so these run without a GPU)."""
    t = _tree()
    v = _verdict()
    big = _cfg(R=64, D=32, V=151936, B=256, K=16)  # about 156 MiB of scratch
    assert lib.tsb_workspace_bytes(ctypes.byref(big)) > tsb.NOALLOC_SCRATCH_BYTES
    assert lib.tsb_step_noalloc(ctypes.byref(big), FAKE, FAKE, 0, FAKE, FAKE, FAKE, ctypes.byref(t), FAKE,
                                ctypes.byref(v), None) == 5
    assert "scratch" in lib.tsb_last_error().decode()
    batched = _cfg(R=16, D=16, V=151936, B=128, K=10)
    assert lib.tsb_workspace_bytes(ctypes.byref(batched)) <= tsb.NOALLOC_SCRATCH_BYTES
    assert lib.tsb_step_noalloc(ctypes.byref(_cfg(K=0)), FAKE, FAKE, 0, FAKE, FAKE, FAKE, ctypes.byref(t), FAKE,
                                ctypes.byref(v), None) == 2
    assert lib.tsb_step_noalloc(ctypes.byref(batched), None, FAKE, 0, FAKE, FAKE, FAKE, ctypes.byref(t), FAKE,
                                ctypes.byref(v), None) == 1
    bad_v = _verdict()
    bad_v.n_acc = None
    assert lib.tsb_step_noalloc(ctypes.byref(batched), FAKE, FAKE, 0, FAKE, FAKE, FAKE, ctypes.byref(t), FAKE,
                                ctypes.byref(bad_v), None) == 1


def test_traversal_entry_points_validate(lib):
    cfg = _cfg()
    need = lib.tsb_workspace_bytes(ctypes.byref(cfg))
    t = _tree()
    v = _verdict()
    assert lib.tsb_verify_traversal(ctypes.byref(_cfg(K=0)), FAKE, FAKE, FAKE, ctypes.byref(t), FAKE, 0,
                                    ctypes.byref(v), FAKE, need, None) == 2
    assert lib.tsb_verify_traversal(ctypes.byref(cfg), FAKE, None, FAKE, ctypes.byref(t), FAKE, 0, ctypes.byref(v),
                                    FAKE, need, None) == 1
    assert lib.tsb_verify_traversal(ctypes.byref(cfg), FAKE, FAKE, FAKE, ctypes.byref(t), FAKE, 0, ctypes.byref(v),
                                    FAKE, need - 1, None) == 5
    assert lib.tsb_step_traversal(ctypes.byref(_cfg(temperature=-2.0)), FAKE, FAKE, 0, FAKE, FAKE, FAKE,
                                  ctypes.byref(t), FAKE, ctypes.byref(v), FAKE, need, None) == 4
    assert lib.tsb_step_traversal(ctypes.byref(cfg), FAKE, FAKE, 0, FAKE, FAKE, FAKE, ctypes.byref(t), None,
                                  ctypes.byref(v), FAKE, need, None) == 1
