"""ctypes binding of libhvd (include/hvd.h): argument marshalling only.

Every step of the verify path runs in the library's HIP kernels.  PyTorch
supplies device memory (borrowed buffers) and the HIP stream.  If the built
library is missing, loading fails loudly; there is no fallback.
"""

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libhvd.so")

HVD_OK, HVD_ERR_ARG, HVD_ERR_STATE, HVD_ERR_OOM, HVD_ERR_RANGE, HVD_ERR_DEVICE = 0, -1, -2, -3, -4, -5
_STATUS = {0: "HVD_OK", -1: "HVD_ERR_ARG", -2: "HVD_ERR_STATE", -3: "HVD_ERR_OOM", -4: "HVD_ERR_RANGE",
           -5: "HVD_ERR_DEVICE"}

EXPORTS = ("hvd_model_bytes", "hvd_model_load", "hvd_model_free", "hvd_kv_bytes", "hvd_kv_alloc", "hvd_kv_free",
           "hvd_prefill", "hvd_verify", "hvd_verify_tree", "hvd_commit", "hvd_truncate", "hvd_seq_free", "hvd_seq_info",
           "hvd_kv_free_pages", "hvd_profile_enable", "hvd_profile_read", "hvd_kv_set_option", "hvd_last_error",
           "hvd_async_begin", "hvd_async_step", "hvd_async_end", "hvd_verify_noalloc", "hvd_flow_trace",
           "hvd_measure_mfma_peak")
HVD_OPT_GRAPHS = 1
HVD_OPT_MLP_SINGLE = 2
HVD_OPT_LM_SINGLE = 3
HVD_OPT_FLOW = 4
HVD_OPT_FLOW_ITEMS = 5
HVD_OPT_ATTN_O = 6
HVD_OPT_GEMM_MIN_BLOCKS = 10
HVD_OPT_ATTN_MIN_ITEMS = 11
HVD_OPT_ATTN_MAX_NP = 12
HVD_OPT_SKINNY_MAX_MT = 13
HVD_OPT_NS8_MT3 = 14
HVD_OPT_PREFILL_ROWS = 15
HVD_OPT_GEMM_SHAPE = 16  # + GEMM family
HVD_OPT_TILED_SHAPE = 24  # + GEMM family
GEMM_FAMILIES = ("qkv", "o", "gateup", "down", "lm")
MAX_TREE_NODES = 63  # nodes per token tree (hvd_verify_tree)


LAYER_TENSORS = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "wg", "wu", "wd")


def tensor_names(n_layers: int):
    """Canonical order of the tensors hvd_model_load takes (include/hvd.h)."""
    return (["embed"] + [f"layers.{l}.{n}" for l in range(n_layers) for n in LAYER_TENSORS]
            + ["final_norm", "lm_head"])


class HvdError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{_STATUS.get(status, status)}: {msg}")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("max_draft", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("max_pos", ctypes.c_int32), ("rope_theta", ctypes.c_float), ("rms_eps", ctypes.c_float)]

    @classmethod
    def from_model_config(cls, c):
        return cls(c.n_layers, c.d_model, c.n_q_heads, c.n_kv_heads, c.head_dim, c.ffn_dim, c.vocab,
                   c.max_draft, c.page_size, c.max_pos, c.rope_theta, c.rms_eps)


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libhvd.so (built by paper_2606_01019_amd.build); raises if absent."""
    global _lib
    if _lib is not None:
        return _lib
    # torch first: it loads its own HIP runtime, which libhvd.so then shares
    # (loaded the other way round, the process would hold two runtimes)
    import torch  # noqa: F401
    if not os.path.exists(path):
        raise RuntimeError(f"libhvd.so not built at {path}: run `python -m paper_2606_01019_amd.build`")
    L = ctypes.CDLL(path)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    PI32 = ctypes.POINTER(ctypes.c_int32)
    sig = {
        "hvd_model_bytes": (SZ, [ctypes.POINTER(Config)]),
        "hvd_model_load": (I32, [ctypes.POINTER(Config), ctypes.POINTER(P), P, SZ, P, ctypes.POINTER(P)]),
        "hvd_model_free": (None, [P]),
        "hvd_kv_bytes": (SZ, [ctypes.POINTER(Config), I32, I32]),
        "hvd_kv_alloc": (I32, [P, I32, I32, P, SZ, P, ctypes.POINTER(P)]),
        "hvd_kv_free": (None, [P]),
        "hvd_prefill": (I32, [P, P, I32, P, I32]),
        "hvd_verify": (I32, [P, P, I32, P, P, P, P, P, P, P]),
        "hvd_verify_noalloc": (I32, [P, P, I32, P, P, P, P, P, P, P]),
        "hvd_verify_tree": (I32, [P, P, I32, P, P, P, P, P, P, P, P, P]),
        "hvd_commit": (I32, [P, P, I32, P, P]),
        "hvd_truncate": (I32, [P, I32, I32, I32]),
        "hvd_seq_free": (I32, [P, I32]),
        "hvd_seq_info": (I32, [P, I32, PI32, PI32, PI32]),
        "hvd_kv_free_pages": (I32, [P]),
        "hvd_profile_enable": (I32, [P, I32]),
        "hvd_profile_read": (I32, [P, I32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64),
                                   ctypes.POINTER(ctypes.c_double)]),
        "hvd_kv_set_option": (I32, [P, I32, I32]),
        "hvd_last_error": (ctypes.c_char_p, []),
        "hvd_async_begin": (I32, [P, P, I32, P, P, P, I32, P, P, P, P, I32, P, ctypes.POINTER(P)]),
        "hvd_async_step": (I32, [P, I32]),
        "hvd_async_end": (I32, [P, PI32]),
        "hvd_flow_trace": (I32, [P, P, ctypes.c_int64]),
        "hvd_measure_mfma_peak": (I32, [P, ctypes.POINTER(ctypes.c_double)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def measure_mfma_peak(stream=None) -> float:
    """Dense fp16 MFMA TFLOP/s measured on the current GPU (hvd_measure_mfma_peak)."""
    t = ctypes.c_double()
    _check(load_library().hvd_measure_mfma_peak(_stream(stream), ctypes.byref(t)))
    return t.value


def _check(status):
    if status != HVD_OK:
        raise HvdError(status, load_library().hvd_last_error().decode())


def _i32(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _ptr(a):
    # the address as an int (the int32-array parameters are declared void*):
    # ctypes' data_as costs microseconds per call on the step's path
    return a.ctypes.data if a is not None and a.size else None


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class Model:
    """Target model on the GPU.  ``tensors`` maps canonical names (see
    workloads.weights) to uint16 bf16 arrays, or is a list in canonical order."""

    def __init__(self, cfg, tensors, names=None, stream=None):
        import torch
        self.lib = load_library()
        self.cfg = cfg
        self.ccfg = Config.from_model_config(cfg)
        if isinstance(tensors, dict):
            arrs = [np.ascontiguousarray(tensors[n], dtype=np.uint16) for n in tensor_names(cfg.n_layers)]
        else:
            arrs = [np.ascontiguousarray(t, dtype=np.uint16) for t in tensors]
        ptrs = (ctypes.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])
        nbytes = self.lib.hvd_model_bytes(ctypes.byref(self.ccfg))
        if nbytes == 0:
            raise HvdError(HVD_ERR_ARG, "unsupported config")
        self.buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        self.stream = stream
        h = ctypes.c_void_p()
        _check(self.lib.hvd_model_load(ctypes.byref(self.ccfg), ptrs, ctypes.c_void_p(self.buf.data_ptr()),
                                       nbytes, _stream(stream), ctypes.byref(h)))
        self.handle = h

    def close(self):
        """Release the handle and the device buffer (no KV cache of this model
        may be used afterwards)."""
        if getattr(self, "handle", None):
            self.lib.hvd_model_free(self.handle)
            self.handle = None
        self.buf = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class KVCache:
    """Paged KV cache plus per-step workspace bound to one Model."""

    def __init__(self, model: Model, max_seqs: int, n_pages: int, stream=None):
        import torch
        self.lib = model.lib
        self.model = model
        nbytes = self.lib.hvd_kv_bytes(ctypes.byref(model.ccfg), max_seqs, n_pages)
        if nbytes == 0:
            raise HvdError(HVD_ERR_ARG, "bad max_seqs / n_pages")
        self.buf = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        torch.cuda.current_stream().synchronize()  # buffer allocated before the library's stream uses it
        # The library's work runs on its own (default-priority) stream: the
        # null stream adds cross-stream synchronization to every launch.
        self.stream = stream if stream is not None else torch.cuda.Stream()
        h = ctypes.c_void_p()
        _check(self.lib.hvd_kv_alloc(model.handle, max_seqs, n_pages, ctypes.c_void_p(self.buf.data_ptr()), nbytes,
                                     _stream(self.stream), ctypes.byref(h)))
        self.handle = h
        self.max_seqs = max_seqs

    # -- calls of the C ABI
    def prefill(self, seq_id: int, tokens):
        t = _i32(tokens)
        _check(self.lib.hvd_prefill(self.model.handle, self.handle, seq_id, _ptr(t), t.size))

    def verify(self, seq_ids, ctx_lens, drafts, logits=None, noalloc=False):
        """drafts: list of 1-D token arrays.  logits: optional torch float32
        CUDA tensor [sum(k+1), vocab].  Returns (accepted, next_token).
        noalloc: call hvd_verify_noalloc (step scratch in the library's
        static device array) instead of hvd_verify."""
        ids = _i32(seq_ids)
        ctx = _i32(ctx_lens)
        lens = _i32([len(d) for d in drafts])
        if len(drafts) == 1:
            flat = _i32(np.asarray(drafts[0]).reshape(-1))
        else:
            flat = _i32(np.concatenate([np.asarray(d, dtype=np.int64).reshape(-1) for d in drafts])
                        if len(drafts) else np.zeros(0))
        acc = np.zeros(ids.size, dtype=np.int32)
        nxt = np.zeros(ids.size, dtype=np.int32)
        lp = None
        if logits is not None:
            rows = int(lens.sum()) + ids.size
            assert logits.is_cuda and logits.dtype.is_floating_point and logits.element_size() == 4
            assert logits.is_contiguous() and logits.numel() >= rows * self.model.cfg.vocab
            lp = ctypes.c_void_p(logits.data_ptr())
        fn = self.lib.hvd_verify_noalloc if noalloc else self.lib.hvd_verify
        _check(fn(self.model.handle, self.handle, ids.size, _ptr(ids), _ptr(ctx), _ptr(flat),
                  _ptr(lens), _ptr(acc), _ptr(nxt), lp))
        return acc, nxt

    def verify_tree(self, seq_ids, ctx_lens, trees, logits=None):
        """trees: list of (node_tokens, node_parents) pairs (parent -1 = the
        pending token, else an earlier node).  logits: optional torch float32
        CUDA tensor [sum(n+1), vocab].  Returns (accepted, next_token,
        accepted node paths as lists)."""
        ids = _i32(seq_ids)
        ctx = _i32(ctx_lens)
        counts = _i32([len(t) for t, _ in trees])
        cat = lambda xs: np.concatenate([np.asarray(x, dtype=np.int64).reshape(-1) for x in xs]) if xs else np.zeros(0)
        toks = _i32(cat([t for t, _ in trees]))
        pars = _i32(cat([p for _, p in trees]))
        acc = np.zeros(ids.size, dtype=np.int32)
        nxt = np.zeros(ids.size, dtype=np.int32)
        paths = np.zeros((ids.size, MAX_TREE_NODES), dtype=np.int32)
        lp = None
        if logits is not None:
            rows = int(counts.sum()) + ids.size
            assert logits.is_cuda and logits.dtype.is_floating_point and logits.element_size() == 4
            assert logits.is_contiguous() and logits.numel() >= rows * self.model.cfg.vocab
            lp = ctypes.c_void_p(logits.data_ptr())
        _check(self.lib.hvd_verify_tree(self.model.handle, self.handle, ids.size, _ptr(ids), _ptr(ctx), _ptr(toks),
                                        _ptr(pars), _ptr(counts), _ptr(acc), _ptr(nxt), _ptr(paths), lp))
        return acc, nxt, [paths[b, :acc[b]].tolist() for b in range(ids.size)]

    def commit(self, seq_ids, keep=None):
        ids = _i32(seq_ids)
        kp = _i32(keep) if keep is not None else None
        _check(self.lib.hvd_commit(self.model.handle, self.handle, ids.size, _ptr(ids), _ptr(kp)))

    def truncate(self, seq_id, new_ctx, pending):
        _check(self.lib.hvd_truncate(self.handle, seq_id, new_ctx, pending))

    def seq_free(self, seq_id):
        _check(self.lib.hvd_seq_free(self.handle, seq_id))

    def seq_info(self, seq_id):
        a, b, c = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        _check(self.lib.hvd_seq_info(self.handle, seq_id, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)))
        return a.value, b.value, bool(c.value)

    def set_mlp_single(self, on):
        """Verify MLP GEMMs on the fp16 activation alone or on the fp16 hi + lo
        pair: True = both GEMMs single, False = both on the pair, or the
        option's value (2 = gate/up single, the default; 3 = down single)."""
        value = (1 if on else 0) if isinstance(on, bool) else int(on)
        _check(self.lib.hvd_kv_set_option(self.handle, HVD_OPT_MLP_SINGLE, value))

    def set_lm_single(self, on: bool):
        """Verify LM head on the fp16 activation alone (default) or on the
        fp16 hi + lo pair."""
        _check(self.lib.hvd_kv_set_option(self.handle, HVD_OPT_LM_SINGLE, 1 if on else 0))

    def set_flow(self, on: bool):
        """One-launch verify step for batches of at most 32 rows, or one
        kernel launch per GEMM / attention pass (the default)."""
        _check(self.lib.hvd_kv_set_option(self.handle, HVD_OPT_FLOW, 1 if on else 0))

    def set_attn_o(self, on: bool):
        """Attention, merge and O projection of small verify batches as one
        launch per layer, or as separate launches (the default)."""
        _check(self.lib.hvd_kv_set_option(self.handle, HVD_OPT_ATTN_O, 1 if on else 0))

    def set_flow_items(self, n: int):
        """Attention work items the one-launch step aims for (tuning)."""
        _check(self.lib.hvd_kv_set_option(self.handle, HVD_OPT_FLOW_ITEMS, int(n)))

    def flow_trace(self, buf=None):
        """Record a per-workgroup timeline of one-launch steps into buf (an
        int64 CUDA tensor, 4 words per workgroup), or stop (None)."""
        if buf is None:
            _check(self.lib.hvd_flow_trace(self.handle, None, 0))
        else:
            assert buf.is_cuda and buf.element_size() == 8 and buf.is_contiguous()
            _check(self.lib.hvd_flow_trace(self.handle, ctypes.c_void_p(buf.data_ptr()), buf.numel()))

    def set_option(self, option: int, value: int):
        """Set one of the handle's launch options (HVD_OPT_*)."""
        _check(self.lib.hvd_kv_set_option(self.handle, int(option), int(value)))

    def set_gemm_shape(self, family: str, strips: int = 0, splits: int = 0):
        """Force the weight-streaming GEMM shape of one GEMM family (strips
        per workgroup, K splits); strips 0 returns it to the policy."""
        value = strips * 100 + splits if strips else 0
        self.set_option(HVD_OPT_GEMM_SHAPE + GEMM_FAMILIES.index(family), value)

    def set_tiled_shape(self, family: str, tile: int = -1, splits: int = 0):
        """Force the tiled GEMM shape of one GEMM family (tile 0..4, K
        splits); tile -1 returns it to the policy."""
        value = (tile + 1) * 100 + splits if tile >= 0 else 0
        self.set_option(HVD_OPT_TILED_SHAPE + GEMM_FAMILIES.index(family), value)

    def set_graphs(self, on: bool):
        """Replay step kernels from cached HIP graphs, or launch eagerly (default)."""
        _check(self.lib.hvd_kv_set_option(self.handle, HVD_OPT_GRAPHS, 1 if on else 0))

    def free_pages(self):
        return self.lib.hvd_kv_free_pages(self.handle)

    def profile_enable(self, on=True):
        _check(self.lib.hvd_profile_enable(self.handle, 1 if on else 0))

    def profile_read(self, family):
        ms, n, b = ctypes.c_double(), ctypes.c_int64(), ctypes.c_double()
        _check(self.lib.hvd_profile_read(self.handle, family, ctypes.byref(ms), ctypes.byref(n), ctypes.byref(b)))
        return ms.value, n.value, b.value

    def async_loop(self, seq_ids, ctx_lens, draft_lens, max_steps, ref=None, ref_start=None):
        """Open a device-resident verify loop (hvd_async_begin); see AsyncLoop."""
        return AsyncLoop(self, seq_ids, ctx_lens, draft_lens, max_steps, ref, ref_start)

    def close(self):
        if getattr(self, "handle", None):
            self.stream.synchronize()
            self.lib.hvd_kv_free(self.handle)
            self.handle = None
        self.buf = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class AsyncLoop:
    """Device-resident verify loop over fixed draft lengths (hvd_async_*).

    Owns the device buffers the library reads and advances: ``drafts``
    (int32 [sum k], the draft tokens of the next step, packed in batch
    order), ``state`` (int32 [2B + 1]: ctx, pending token, steps done) and
    ``history`` (int32 [max_steps, B, 2]: accepted length and next token of
    every step).  A GPU drafter writes ``drafts`` on ``kv.stream`` between
    steps; with ``ref`` (int32 CUDA tensor [B, ref_len]) and ``ref_start``
    the library's copy drafter fills them from that token stream instead.
    ``step(n)`` only enqueues; ``end()`` waits and hands the sequences back to
    the host-side calls."""

    def __init__(self, kv, seq_ids, ctx_lens, draft_lens, max_steps, ref=None, ref_start=None):
        import torch
        self.kv = kv
        self.lib = kv.lib
        ids, ctx, lens = _i32(seq_ids), _i32(ctx_lens), _i32(draft_lens)
        B = ids.size
        self.draft_lens = lens
        self.drafts = torch.zeros(max(1, int(lens.sum())), dtype=torch.int32, device="cuda")
        self.state = torch.zeros(2 * B + 1, dtype=torch.int32, device="cuda")
        self.history = torch.zeros((max(1, max_steps), B, 2), dtype=torch.int32, device="cuda")
        self.ref = None
        rs = None
        ref_len = 0
        if ref is not None:
            assert ref.is_cuda and ref.dtype == torch.int32 and ref.dim() == 2 and ref.shape[0] == B
            self.ref = ref.contiguous()
            ref_len = int(self.ref.shape[1])
            rs = _i32(ref_start)
        torch.cuda.current_stream().synchronize()  # buffers exist before the library's stream uses them
        h = ctypes.c_void_p()
        vp = lambda t: ctypes.c_void_p(t.data_ptr()) if t is not None else None
        _check(self.lib.hvd_async_begin(kv.model.handle, kv.handle, B, _ptr(ids), _ptr(ctx), _ptr(lens), max_steps,
                                        vp(self.drafts), vp(self.state), vp(self.history), vp(self.ref), ref_len,
                                        _ptr(rs), ctypes.byref(h)))
        self.handle = h
        self.steps_done = 0

    def step(self, n: int = 1):
        _check(self.lib.hvd_async_step(self.handle, n))

    def end(self):
        """Wait for the enqueued steps, return the host-side calls their
        sequences; returns the number of steps run."""
        if getattr(self, "handle", None):
            n = ctypes.c_int32()
            h, self.handle = self.handle, None
            _check(self.lib.hvd_async_end(h, ctypes.byref(n)))
            self.steps_done = n.value
        return self.steps_done

    def __del__(self):
        try:
            self.end()
        except Exception:
            pass
