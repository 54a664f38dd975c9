"""Python binding of the gfx950 tree-replay library (libtsubame.so).

Argument marshalling only: every stage of a round (plan, replay, verify)
runs in the HIP kernels behind the C ABI of include/tsubame.h. PyTorch
supplies device memory and the stream. There is no CPU fallback: if the
library is not built, or a call fails, an exception is raised.

Entry points mirror the C ABI: plan, plan_ep, replay, verify, step, workspace_bytes,
verify_traversal, step_traversal (traversal verification), step_noalloc,
the First + Naive baseline: first_tokens, verify_naive, step_first, and the
round over sparse candidate pools with context-dependent draft distributions:
pool_plan, pool_replay, pool_verify, pool_step, pool_workspace_bytes.
`Round` bundles the output buffers of one configuration.
"""
import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtsubame.so")

TSB_F32 = 0
TSB_BF16 = 1
REQ_NONFINITE = 1
REQ_DEGENERATE_RESIDUAL = 2
REQ_BUDGET_SHORT = 4
REQ_WALK_TIMEOUT = 8
REQ_BAD_TOKEN = 16
REQ_BAD_TREE = 32
POOL_MAX = 64
FLAG_NO_PRUNE = 1
FLAG_READ_ROWS = 2
FLAG_STREAM_ROWS = 4
MAX_D, MAX_K, MAX_B, TRACE_MAX = 64, 32, 1023, 256
KERNELS = ("draft_partials", "plan_tree", "replay_scan", "replay_merge", "target_partials",
           "verify_walk", "verify_naive", "pool_partials", "pool_lists", "pool_plan", "pool_replay", "pool_walk",
           "traversal_walk", "scan_target")

EXPORTS = ("tsb_workspace_bytes", "tsb_plan", "tsb_plan_ep", "tsb_replay", "tsb_verify", "tsb_step",
           "tsb_first_tokens", "tsb_verify_naive", "tsb_step_first",
           "tsb_pool_workspace_bytes", "tsb_pool_plan", "tsb_pool_replay", "tsb_pool_verify", "tsb_pool_step",
           "tsb_status_string", "tsb_last_error", "tsb_version", "tsb_profile_kernel", "tsb_step_noalloc",
           "tsb_verify_traversal", "tsb_step_traversal", "tsb_stats_enable", "tsb_stats_read")
NOALLOC_SCRATCH_BYTES = 32 << 20


class TsbConfig(ctypes.Structure):
    _fields_ = [("R", ctypes.c_int32), ("D", ctypes.c_int32), ("V", ctypes.c_int32), ("B", ctypes.c_int32),
                ("K", ctypes.c_int32), ("temperature", ctypes.c_float), ("dtype", ctypes.c_uint32),
                ("flags", ctypes.c_uint32), ("seed", ctypes.c_uint64)]


class TsbTree(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("parent", "depth", "rank", "n_children", "first_child",
                                               "score", "n_nodes", "plan_margin")]


STATS_FIELDS = ("replay_items", "replay_tokens", "replay_groups_live", "replay_groups_keyed", "walk_requests",
                "walk_nodes", "walk_tests", "walk_exchanges", "plan_requests", "plan_merge_ticks",
                "plan_search_ticks", "plan_emit_ticks", "plan_rounds")


class TsbStats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in STATS_FIELDS] + [("reserved", ctypes.c_uint64 * 3)]


class TsbVerdict(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("n_acc", "acc_node", "acc_tok", "bonus", "req_status",
                                               "target_lse", "trace")]


class TsbError(RuntimeError):
    def __init__(self, status, where):
        lib = load()
        msg = "%s failed: %s (%s)" % (where, lib.tsb_status_string(status).decode(),
                                      lib.tsb_last_error().decode())
        super().__init__(msg)
        self.status = status


_LIB = None


def load(path=LIB_PATH):
    """Load libtsubame.so (raises if it has not been built)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise ImportError("libtsubame.so is not built (run paper_2609_33652_amd/build.py or "
                          "__graft_entry__.build()); there is no fallback path")
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    lib.tsb_workspace_bytes.restype = ctypes.c_size_t
    lib.tsb_workspace_bytes.argtypes = [ctypes.POINTER(TsbConfig)]
    lib.tsb_plan.restype = ctypes.c_int
    lib.tsb_plan.argtypes = [ctypes.POINTER(TsbConfig), P, P, P, P, ctypes.POINTER(TsbTree), P, P,
                             ctypes.c_size_t, P]
    lib.tsb_plan_ep.restype = ctypes.c_int
    lib.tsb_plan_ep.argtypes = [ctypes.POINTER(TsbConfig), ctypes.c_int32, P, P, P, P, ctypes.POINTER(TsbTree), P, P,
                                ctypes.c_size_t, P]
    lib.tsb_replay.restype = ctypes.c_int
    lib.tsb_replay.argtypes = [ctypes.POINTER(TsbConfig), P, P, ctypes.POINTER(TsbTree), ctypes.c_uint32, P, P,
                               ctypes.c_size_t, P]
    lib.tsb_verify.restype = ctypes.c_int
    lib.tsb_verify.argtypes = [ctypes.POINTER(TsbConfig), P, P, P, ctypes.POINTER(TsbTree), P, ctypes.c_uint32,
                               ctypes.POINTER(TsbVerdict), P, ctypes.c_size_t, P]
    lib.tsb_step.restype = ctypes.c_int
    lib.tsb_step.argtypes = [ctypes.POINTER(TsbConfig), P, P, ctypes.c_uint32, P, P, P, ctypes.POINTER(TsbTree), P,
                             ctypes.POINTER(TsbVerdict), P, ctypes.c_size_t, P]
    lib.tsb_first_tokens.restype = ctypes.c_int
    lib.tsb_first_tokens.argtypes = [ctypes.POINTER(TsbConfig), P, ctypes.POINTER(TsbTree), P, P]
    lib.tsb_verify_naive.restype = ctypes.c_int
    lib.tsb_verify_naive.argtypes = [ctypes.POINTER(TsbConfig), P, ctypes.POINTER(TsbTree), P, ctypes.c_uint32,
                                     ctypes.POINTER(TsbVerdict), P, ctypes.c_size_t, P]
    lib.tsb_verify_traversal.restype = ctypes.c_int
    lib.tsb_verify_traversal.argtypes = lib.tsb_verify.argtypes
    lib.tsb_step_traversal.restype = ctypes.c_int
    lib.tsb_step_traversal.argtypes = lib.tsb_step.argtypes
    lib.tsb_step_noalloc.restype = ctypes.c_int
    lib.tsb_step_noalloc.argtypes = [ctypes.POINTER(TsbConfig), P, P, ctypes.c_uint32, P, P, P,
                                     ctypes.POINTER(TsbTree), P, ctypes.POINTER(TsbVerdict), P]
    lib.tsb_step_first.restype = ctypes.c_int
    lib.tsb_step_first.argtypes = lib.tsb_step.argtypes
    I = ctypes.c_int32
    cfgp, treep, verdp = ctypes.POINTER(TsbConfig), ctypes.POINTER(TsbTree), ctypes.POINTER(TsbVerdict)
    lib.tsb_pool_workspace_bytes.restype = ctypes.c_size_t
    lib.tsb_pool_workspace_bytes.argtypes = [cfgp, I]
    lib.tsb_pool_plan.restype = ctypes.c_int
    lib.tsb_pool_plan.argtypes = [cfgp, I, P, P, P, treep, P, P, P, ctypes.c_size_t, P]
    lib.tsb_pool_replay.restype = ctypes.c_int
    lib.tsb_pool_replay.argtypes = [cfgp, I, P, P, P, treep, ctypes.c_uint32, P, P]
    lib.tsb_pool_verify.restype = ctypes.c_int
    lib.tsb_pool_verify.argtypes = [cfgp, I, P, P, P, P, treep, P, ctypes.c_uint32, verdp, P, ctypes.c_size_t, P]
    lib.tsb_pool_step.restype = ctypes.c_int
    lib.tsb_pool_step.argtypes = [cfgp, I, P, P, P, ctypes.c_uint32, P, treep, P, verdp, P, ctypes.c_size_t, P]
    lib.tsb_status_string.restype = ctypes.c_char_p
    lib.tsb_status_string.argtypes = [ctypes.c_int]
    lib.tsb_last_error.restype = ctypes.c_char_p
    lib.tsb_last_error.argtypes = []
    lib.tsb_version.restype = ctypes.c_int32
    lib.tsb_version.argtypes = []
    lib.tsb_profile_kernel.restype = ctypes.c_int
    lib.tsb_profile_kernel.argtypes = [ctypes.c_int32, P, P]
    lib.tsb_stats_enable.restype = ctypes.c_int
    lib.tsb_stats_enable.argtypes = [ctypes.c_int32]
    lib.tsb_stats_read.restype = ctypes.c_int
    lib.tsb_stats_read.argtypes = [ctypes.POINTER(TsbStats), ctypes.c_int32]
    _LIB = lib
    return lib


def walk_reads_rows(cfg):
    """Whether the WoR-RRS walk of cfg reads each target row as it enters the row's node (the library's
    rule: the flags, else more than 128 MiB of target); the other way streams every row first."""
    if cfg.flags & FLAG_READ_ROWS:
        return True
    if cfg.flags & FLAG_STREAM_ROWS:
        return False
    return cfg.R * (cfg.B + 1) * cfg.V * (2 if cfg.dtype == TSB_BF16 else 4) > (128 << 20)


def make_config(R, D, V, B, K, temperature, dtype, seed, flags=0):
    dt = {"f32": TSB_F32, "bf16": TSB_BF16, TSB_F32: TSB_F32, TSB_BF16: TSB_BF16}.get(dtype, dtype)
    return TsbConfig(R=int(R), D=int(D), V=int(V), B=int(B), K=int(K), temperature=float(temperature),
                     dtype=int(dt), flags=int(flags), seed=int(seed) & 0xFFFFFFFFFFFFFFFF)


def workspace_bytes(cfg):
    return int(load().tsb_workspace_bytes(ctypes.byref(cfg)))


def pool_workspace_bytes(cfg, P):
    return int(load().tsb_pool_workspace_bytes(ctypes.byref(cfg), int(P)))


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


_LOGIT_DTYPES = {TSB_F32: torch.float32, TSB_BF16: torch.bfloat16}


def _check(t, shape, dtype, name):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch tensor" % name)
    if t.device.type != "cuda":
        raise ValueError("%s must be a device tensor" % name)
    if tuple(t.shape) != tuple(shape) or t.dtype != dtype or not t.is_contiguous():
        raise ValueError("%s must be a contiguous %s tensor of shape %s (got %s %s)"
                         % (name, dtype, tuple(shape), t.dtype, tuple(t.shape)))


class Round:
    """Output buffers and workspace of one configuration on one device."""

    def __init__(self, cfg, device="cuda", target_lse=False, trace=False, pool=None):
        """pool: pool size P to also hold the buffers of the pool entry points."""
        self.cfg = cfg
        self.pool = None if pool is None else int(pool)
        R, D, B, K = cfg.R, cfg.D, cfg.B, cfg.K
        dev = torch.device(device)
        i32, f64 = torch.int32, torch.float64
        self.draft_lse = torch.empty(R, D, dtype=f64, device=dev)
        self.topk_tok = torch.empty(R, D, K, dtype=i32, device=dev)
        self.topk_lp = torch.empty(R, D, K, dtype=torch.float32, device=dev)
        self.tree = {n: torch.empty(R, B + 1, dtype=i32, device=dev)
                     for n in ("parent", "depth", "rank", "n_children", "first_child")}
        self.tree["score"] = torch.empty(R, B + 1, dtype=f64, device=dev)
        self.tree["n_nodes"] = torch.empty(R, dtype=i32, device=dev)
        self.tree["plan_margin"] = torch.empty(R, dtype=f64, device=dev)
        self.node_tok = torch.empty(R, B + 1, dtype=i32, device=dev)
        self.n_acc = torch.empty(R, dtype=i32, device=dev)
        self.acc_node = torch.empty(R, D, dtype=i32, device=dev)
        self.acc_tok = torch.empty(R, D, dtype=i32, device=dev)
        self.bonus = torch.empty(R, dtype=i32, device=dev)
        self.req_status = torch.empty(R, dtype=i32, device=dev)
        self.target_lse = torch.empty(R, B + 1, dtype=f64, device=dev) if target_lse else None
        self.trace = torch.empty(R, TRACE_MAX, 4, dtype=f64, device=dev) if trace else None
        nb = workspace_bytes(cfg)
        if nb == 0:
            raise ValueError("invalid configuration")
        self.pool_tok = self.plan_tok = None
        if self.pool is not None:
            nbp = pool_workspace_bytes(cfg, self.pool)
            if nbp == 0:
                raise ValueError("invalid pool size %d" % self.pool)
            nb = max(nb, nbp)
            self.pool_tok = torch.empty(R, D, self.pool, dtype=i32, device=dev)
            self.plan_tok = torch.empty(R, B + 1, dtype=i32, device=dev)
        self.ws = torch.empty(nb + 256, dtype=torch.uint8, device=dev)  # no initial content needed
        off = (-self.ws.data_ptr()) % 256
        self.ws_ptr = ctypes.c_void_p(self.ws.data_ptr() + off)
        self.ws_bytes = nb
        self._tree_c = TsbTree(**{k: v.data_ptr() for k, v in self.tree.items()})
        self._verdict_c = TsbVerdict(n_acc=self.n_acc.data_ptr(), acc_node=self.acc_node.data_ptr(),
                                     acc_tok=self.acc_tok.data_ptr(), bonus=self.bonus.data_ptr(),
                                     req_status=self.req_status.data_ptr(),
                                     target_lse=self.target_lse.data_ptr() if target_lse else None,
                                     trace=self.trace.data_ptr() if trace else None)

    # ---------------------------------------------------------------- inputs
    def _logits(self, t, rows, name):
        cfg = self.cfg
        _check(t, (cfg.R, rows, cfg.V), _LOGIT_DTYPES[cfg.dtype], name)

    def load_tree(self, tree):
        """Copy a topology (dict of [R, B+1] / [R] tensors) into the buffers."""
        for k, v in tree.items():
            if k in self.tree:
                self.tree[k].copy_(v)

    # ---------------------------------------------------------------- stages
    def plan(self, draft, stream=None):
        self._logits(draft, self.cfg.D, "draft")
        st = load().tsb_plan(ctypes.byref(self.cfg), _ptr(draft), _ptr(self.draft_lse), _ptr(self.topk_tok),
                             _ptr(self.topk_lp), ctypes.byref(self._tree_c), _ptr(self.req_status), self.ws_ptr,
                             self.ws_bytes, _stream(stream))
        if st:
            raise TsbError(st, "tsb_plan")

    def plan_ep(self, draft, frontier, stream=None):
        """First pass by expand-then-prune with the given frontier width."""
        self._logits(draft, self.cfg.D, "draft")
        st = load().tsb_plan_ep(ctypes.byref(self.cfg), int(frontier), _ptr(draft), _ptr(self.draft_lse),
                                _ptr(self.topk_tok), _ptr(self.topk_lp), ctypes.byref(self._tree_c),
                                _ptr(self.req_status), self.ws_ptr, self.ws_bytes, _stream(stream))
        if st:
            raise TsbError(st, "tsb_plan_ep")

    def replay(self, draft, step, stream=None):
        self._logits(draft, self.cfg.D, "draft")
        st = load().tsb_replay(ctypes.byref(self.cfg), _ptr(draft), _ptr(self.topk_tok), ctypes.byref(self._tree_c),
                               int(step) & 0xFFFFFFFF, _ptr(self.node_tok), self.ws_ptr, self.ws_bytes,
                               _stream(stream))
        if st:
            raise TsbError(st, "tsb_replay")

    def verify(self, draft, target, step, stream=None):
        self._logits(draft, self.cfg.D, "draft")
        self._logits(target, self.cfg.B + 1, "target")
        st = load().tsb_verify(ctypes.byref(self.cfg), _ptr(draft), _ptr(self.draft_lse), _ptr(target),
                               ctypes.byref(self._tree_c), _ptr(self.node_tok), int(step) & 0xFFFFFFFF,
                               ctypes.byref(self._verdict_c), self.ws_ptr, self.ws_bytes, _stream(stream))
        if st:
            raise TsbError(st, "tsb_verify")

    def step(self, draft, target, step, stream=None):
        self._logits(draft, self.cfg.D, "draft")
        self._logits(target, self.cfg.B + 1, "target")
        st = load().tsb_step(ctypes.byref(self.cfg), _ptr(draft), _ptr(target), int(step) & 0xFFFFFFFF,
                             _ptr(self.draft_lse), _ptr(self.topk_tok), _ptr(self.topk_lp),
                             ctypes.byref(self._tree_c), _ptr(self.node_tok), ctypes.byref(self._verdict_c),
                             self.ws_ptr, self.ws_bytes, _stream(stream))
        if st:
            raise TsbError(st, "tsb_step")

    def verify_traversal(self, draft, target, step, stream=None):
        """Traversal verification of the replayed tree (instead of WoR-RRS)."""
        self._logits(draft, self.cfg.D, "draft")
        self._logits(target, self.cfg.B + 1, "target")
        st = load().tsb_verify_traversal(ctypes.byref(self.cfg), _ptr(draft), _ptr(self.draft_lse), _ptr(target),
                                         ctypes.byref(self._tree_c), _ptr(self.node_tok), int(step) & 0xFFFFFFFF,
                                         ctypes.byref(self._verdict_c), self.ws_ptr, self.ws_bytes, _stream(stream))
        if st:
            raise TsbError(st, "tsb_verify_traversal")

    def step_traversal(self, draft, target, step, stream=None):
        self._logits(draft, self.cfg.D, "draft")
        self._logits(target, self.cfg.B + 1, "target")
        st = load().tsb_step_traversal(ctypes.byref(self.cfg), _ptr(draft), _ptr(target), int(step) & 0xFFFFFFFF,
                                       _ptr(self.draft_lse), _ptr(self.topk_tok), _ptr(self.topk_lp),
                                       ctypes.byref(self._tree_c), _ptr(self.node_tok), ctypes.byref(self._verdict_c),
                                       self.ws_ptr, self.ws_bytes, _stream(stream))
        if st:
            raise TsbError(st, "tsb_step_traversal")

    def step_noalloc(self, draft, target, step, stream=None):
        """tsb_step with the library's own per-device scratch instead of this Round's workspace."""
        self._logits(draft, self.cfg.D, "draft")
        self._logits(target, self.cfg.B + 1, "target")
        st = load().tsb_step_noalloc(ctypes.byref(self.cfg), _ptr(draft), _ptr(target), int(step) & 0xFFFFFFFF,
                                     _ptr(self.draft_lse), _ptr(self.topk_tok), _ptr(self.topk_lp),
                                     ctypes.byref(self._tree_c), _ptr(self.node_tok), ctypes.byref(self._verdict_c),
                                     _stream(stream))
        if st:
            raise TsbError(st, "tsb_step_noalloc")

    # ------------------------------------------------- First + Naive baseline
    def first_tokens(self, stream=None):
        """node_tok <- planning candidates of the first-pass tree (needs plan() first)."""
        st = load().tsb_first_tokens(ctypes.byref(self.cfg), _ptr(self.topk_tok), ctypes.byref(self._tree_c),
                                     _ptr(self.node_tok), _stream(stream))
        if st:
            raise TsbError(st, "tsb_first_tokens")

    def verify_naive(self, target, step, stream=None):
        self._logits(target, self.cfg.B + 1, "target")
        st = load().tsb_verify_naive(ctypes.byref(self.cfg), _ptr(target), ctypes.byref(self._tree_c),
                                     _ptr(self.node_tok), int(step) & 0xFFFFFFFF, ctypes.byref(self._verdict_c),
                                     self.ws_ptr, self.ws_bytes, _stream(stream))
        if st:
            raise TsbError(st, "tsb_verify_naive")

    def step_first(self, draft, target, step, stream=None):
        self._logits(draft, self.cfg.D, "draft")
        self._logits(target, self.cfg.B + 1, "target")
        st = load().tsb_step_first(ctypes.byref(self.cfg), _ptr(draft), _ptr(target), int(step) & 0xFFFFFFFF,
                                   _ptr(self.draft_lse), _ptr(self.topk_tok), _ptr(self.topk_lp),
                                   ctypes.byref(self._tree_c), _ptr(self.node_tok), ctypes.byref(self._verdict_c),
                                   self.ws_ptr, self.ws_bytes, _stream(stream))
        if st:
            raise TsbError(st, "tsb_step_first")

    # ------------------------------------------------------------- pools
    def _trans(self, trans):
        cfg = self.cfg
        if cfg.D == 1 and trans is None:
            return None
        _check(trans, (cfg.R, cfg.D - 1, self.pool, self.pool), torch.float32, "trans")
        return trans

    def pool_plan(self, draft, trans, plan_tokens=True, stream=None):
        """First pass over pools of P tokens; plan_tok receives the planning tokens."""
        self._logits(draft, self.cfg.D, "draft")
        tr = self._trans(trans)
        st = load().tsb_pool_plan(ctypes.byref(self.cfg), self.pool, _ptr(draft), _ptr(tr), _ptr(self.pool_tok),
                                  ctypes.byref(self._tree_c), _ptr(self.plan_tok if plan_tokens else None),
                                  _ptr(self.req_status), self.ws_ptr, self.ws_bytes, _stream(stream))
        if st:
            raise TsbError(st, "tsb_pool_plan")

    def pool_replay(self, draft, trans, step, stream=None):
        self._logits(draft, self.cfg.D, "draft")
        tr = self._trans(trans)
        st = load().tsb_pool_replay(ctypes.byref(self.cfg), self.pool, _ptr(draft), _ptr(tr), _ptr(self.pool_tok),
                                    ctypes.byref(self._tree_c), int(step) & 0xFFFFFFFF, _ptr(self.node_tok),
                                    _stream(stream))
        if st:
            raise TsbError(st, "tsb_pool_replay")

    def pool_verify(self, draft, trans, target, step, stream=None):
        self._logits(draft, self.cfg.D, "draft")
        self._logits(target, self.cfg.B + 1, "target")
        tr = self._trans(trans)
        st = load().tsb_pool_verify(ctypes.byref(self.cfg), self.pool, _ptr(draft), _ptr(tr), _ptr(self.pool_tok),
                                    _ptr(target), ctypes.byref(self._tree_c), _ptr(self.node_tok),
                                    int(step) & 0xFFFFFFFF, ctypes.byref(self._verdict_c), self.ws_ptr,
                                    self.ws_bytes, _stream(stream))
        if st:
            raise TsbError(st, "tsb_pool_verify")

    def pool_step(self, draft, trans, target, step, stream=None):
        self._logits(draft, self.cfg.D, "draft")
        self._logits(target, self.cfg.B + 1, "target")
        tr = self._trans(trans)
        st = load().tsb_pool_step(ctypes.byref(self.cfg), self.pool, _ptr(draft), _ptr(tr), _ptr(target),
                                  int(step) & 0xFFFFFFFF, _ptr(self.pool_tok), ctypes.byref(self._tree_c),
                                  _ptr(self.node_tok), ctypes.byref(self._verdict_c), self.ws_ptr, self.ws_bytes,
                                  _stream(stream))
        if st:
            raise TsbError(st, "tsb_pool_step")

    # ---------------------------------------------------------------- results
    def host(self):
        """Copy every output to host memory (synchronises the current stream)."""
        out = {k: v.cpu() for k, v in self.tree.items()}
        for k in ("draft_lse", "topk_tok", "topk_lp", "node_tok", "n_acc", "acc_node", "acc_tok", "bonus",
                  "req_status", "target_lse", "trace", "pool_tok", "plan_tok"):
            v = getattr(self, k)
            out[k] = v.cpu() if v is not None else None
        return out


def profile_kernel(kernel, start=None, stop=None):
    """Bracket later launches of `kernel` (name or id) with the two torch.cuda.Events; None clears."""
    kid = KERNELS.index(kernel) if isinstance(kernel, str) else int(kernel)
    if start is None:
        st = load().tsb_profile_kernel(-1, None, None)
    else:
        st = load().tsb_profile_kernel(kid, ctypes.c_void_p(start.cuda_event), ctypes.c_void_p(stop.cuda_event))
    if st:
        raise TsbError(st, "tsb_profile_kernel")


def stats_enable(on=True):
    """Turn the work counters of the replay scan, the walk and the planner on or off (calling thread)."""
    st = load().tsb_stats_enable(1 if on else 0)
    if st:
        raise TsbError(st, "tsb_stats_enable")


def stats_read(reset=True):
    """The current device's work counters as a dict (waits for the device); reset zeroes them."""
    out = TsbStats()
    st = load().tsb_stats_read(ctypes.byref(out), 1 if reset else 0)
    if st:
        raise TsbError(st, "tsb_stats_read")
    return {n: int(getattr(out, n)) for n in STATS_FIELDS}
