"""ctypes binding of libllmcad (the C ABI in include/llmcad.h).

Argument marshalling only: every step of a pass runs in the library's HIP
kernels.  Device buffers are torch tensors on a ROCm device (torch provides
memory and streams); tree arrays are host int32 arrays.  Importing this module
fails loudly if the library has not been built.
"""

import ctypes
import os

import numpy as np
import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libllmcad.so")

OK = 0
EARG = -1
ETREE = -2
ECAPACITY = -3
ESHAPE = -4
EHIP = -5
EWORKSPACE = -6
MAX_NODES = 128

SYMBOLS = (
    "llmcad_check_config",
    "llmcad_packed_bytes",
    "llmcad_pack_globals",
    "llmcad_pack_layer",
    "llmcad_pack_layer_q4",
    "llmcad_workspace_bytes",
    "llmcad_workspace_init",
    "llmcad_verify_tree",
    "llmcad_verify_tree_noalloc",
    "llmcad_prefill",
    "llmcad_commit_path",
    "llmcad_extend_tree",
    "llmcad_extend_tree_candidates",
    "llmcad_status_string",
    "llmcad_workspace_region",
    "llmcad_timing_enable",
    "llmcad_timing_read",
)

KERNEL_PASS = 0  # the whole pass is one persistent launch


class LlmcadConfig(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32),
        ("d_model", ctypes.c_int32),
        ("n_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("d_ffn", ctypes.c_int32),
        ("vocab", ctypes.c_int32),
        ("rms_eps", ctypes.c_float),
        ("rope_theta", ctypes.c_float),
        ("weight_bits", ctypes.c_int32),
    ]


class LlmcadLayerWeights(ctypes.Structure):
    _fields_ = [(name, ctypes.c_void_p) for name in
                ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down")]


class LlmcadQ4Matrix(ctypes.Structure):
    _fields_ = [("codes", ctypes.c_void_p), ("scales", ctypes.c_void_p)]


class LlmcadQ4LayerWeights(ctypes.Structure):
    _fields_ = [("attn_norm", ctypes.c_void_p), ("w_qkv", LlmcadQ4Matrix), ("w_o", LlmcadQ4Matrix),
                ("ffn_norm", ctypes.c_void_p), ("w_gate_up", LlmcadQ4Matrix), ("w_down", LlmcadQ4Matrix)]


Q4_GROUP = 128  # inputs per scale group of a 4-bit matrix


class LlmcadError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} ({status})")


# Device pass status (workspace region 5), written by the pass kernel.
PASS_OK = 0
PASS_WAIT_TIMEOUT = 1   # a wait of the single-launch pass ran out of its bounded spin
PASS_BAD_PARAMS = 3     # the kernel did not find its parameter block; it did nothing
_PASS_TEXT = {PASS_WAIT_TIMEOUT: "a grid or join wait ran out of its bounded spin (outputs invalid)",
              PASS_BAD_PARAMS: "the kernel did not find its parameter block (nothing computed)"}


class LlmcadPassError(RuntimeError):
    """A pass ended with a non-zero device status: its outputs are invalid."""

    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: device pass status {status}: {_PASS_TEXT.get(status, 'unknown')}")


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(
            f"{_LIB_PATH} is missing: build it with `python -m paper_2309_04255_amd.build` "
            "(there is no fallback implementation)")
    lib = ctypes.CDLL(_LIB_PATH)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    CFG = ctypes.POINTER(LlmcadConfig)
    I32P = ctypes.POINTER(ctypes.c_int32)
    sig = {
        "llmcad_check_config": (ctypes.c_int, [CFG]),
        "llmcad_packed_bytes": (SZ, [CFG]),
        "llmcad_pack_globals": (ctypes.c_int, [CFG, P, P, P, P, SZ, P]),
        "llmcad_pack_layer": (ctypes.c_int, [CFG, I32, ctypes.POINTER(LlmcadLayerWeights), P, SZ, P]),
        "llmcad_pack_layer_q4": (ctypes.c_int, [CFG, I32, ctypes.POINTER(LlmcadQ4LayerWeights), P, SZ, P]),
        "llmcad_workspace_bytes": (SZ, [CFG, I32]),
        "llmcad_workspace_init": (ctypes.c_int, [CFG, I32, P, SZ, P]),
        "llmcad_verify_tree": (ctypes.c_int, [CFG, P, P, P, I32, I32, I32P, I32P, I32, P, P, P, P,
                                              P, SZ, P]),
        "llmcad_verify_tree_noalloc": (ctypes.c_int, [CFG, P, P, P, I32, I32, I32P, I32P, I32, P, P, P, P,
                                                      P, P]),
        "llmcad_prefill": (ctypes.c_int, [CFG, P, P, P, I32, I32P, I32, I32, P, P, SZ, P]),
        "llmcad_commit_path": (ctypes.c_int, [CFG, P, P, I32, I32, P, P, I32, P]),
        "llmcad_extend_tree": (ctypes.c_int, [CFG, P, P, P, I32, I32, I32P, I32P, I32, I32, P, P, SZ, P]),
        "llmcad_extend_tree_candidates": (ctypes.c_int, [CFG, P, P, P, I32, I32, I32P, I32P, I32, I32, ctypes.c_float,
                                                         P, P, P, SZ, P]),
        "llmcad_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "llmcad_workspace_region": (ctypes.c_int, [CFG, I32, I32, ctypes.POINTER(SZ),
                                                   ctypes.POINTER(SZ)]),
        "llmcad_timing_enable": (ctypes.c_int, [I32, I32]),
        "llmcad_timing_read": (ctypes.c_int, [I32, ctypes.POINTER(ctypes.c_double), I32P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


def lib():
    return _lib


def status_string(status: int) -> str:
    return _lib.llmcad_status_string(int(status)).decode()


def make_config(shape) -> LlmcadConfig:
    """From any object with n_layers, d_model, n_heads, head_dim, d_ffn, vocab, rms_eps, rope_theta
    (and optionally weight_bits: 16, the default, or 4)."""
    return LlmcadConfig(shape.n_layers, shape.d_model, shape.n_heads, shape.head_dim, shape.d_ffn,
                        shape.vocab, float(shape.rms_eps), float(shape.rope_theta),
                        int(getattr(shape, "weight_bits", 16)))


def _ptr(t):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _i32(a):
    a = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _check(rc, what):
    if rc != OK:
        raise LlmcadError(rc, what)


def check_config(cfg: LlmcadConfig) -> int:
    return _lib.llmcad_check_config(ctypes.byref(cfg))


def packed_bytes(cfg: LlmcadConfig) -> int:
    return _lib.llmcad_packed_bytes(ctypes.byref(cfg))


def workspace_bytes(cfg: LlmcadConfig, max_n: int) -> int:
    return _lib.llmcad_workspace_bytes(ctypes.byref(cfg), int(max_n))


def pack_globals(cfg, tok_embed, final_norm, lm_head, packed, stream=None):
    _check(_lib.llmcad_pack_globals(ctypes.byref(cfg), _ptr(tok_embed), _ptr(final_norm),
                                    _ptr(lm_head), _ptr(packed), packed.numel() * packed.element_size(),
                                    _stream(stream)), "llmcad_pack_globals")


def pack_layer(cfg, layer: int, w: dict, packed, stream=None):
    src = LlmcadLayerWeights(*(w[k].data_ptr() for k in
                               ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down")))
    _check(_lib.llmcad_pack_layer(ctypes.byref(cfg), int(layer), ctypes.byref(src), _ptr(packed),
                                  packed.numel() * packed.element_size(), _stream(stream)),
           "llmcad_pack_layer")


def pack_layer_q4(cfg, layer: int, w: dict, packed, stream=None):
    """w: attn_norm, ffn_norm (bf16 [d]) and, per matrix m in w_qkv, w_o, w_gate_up,
    w_down, a pair (codes uint8 [out][in/2], scales bf16 [out][in/128]) on the device."""
    def mat(k):
        codes, scales = w[k]
        return LlmcadQ4Matrix(codes.data_ptr(), scales.data_ptr())

    src = LlmcadQ4LayerWeights(w["attn_norm"].data_ptr(), mat("w_qkv"), mat("w_o"), w["ffn_norm"].data_ptr(),
                               mat("w_gate_up"), mat("w_down"))
    _check(_lib.llmcad_pack_layer_q4(ctypes.byref(cfg), int(layer), ctypes.byref(src), _ptr(packed),
                                     packed.numel() * packed.element_size(), _stream(stream)),
           "llmcad_pack_layer_q4")


def workspace_init(cfg, max_n: int, workspace, stream=None):
    _check(_lib.llmcad_workspace_init(ctypes.byref(cfg), int(max_n), _ptr(workspace),
                                      workspace.numel() * workspace.element_size(), _stream(stream)),
           "llmcad_workspace_init")


def verify_tree(cfg, packed, k_cache, v_cache, prefix_len: int, tree_tokens, parent, logits, path,
                accept_len, next_token, workspace, stream=None, raise_on_error=True) -> int:
    """Enqueue one verification pass; returns the status (raises on error by default)."""
    tok, tok_p = _i32(tree_tokens)
    par, par_p = _i32(parent)
    n = len(tok)
    if len(par) != n:
        raise ValueError("tree_tokens and parent differ in length")
    cap = k_cache.shape[-2]
    rc = _lib.llmcad_verify_tree(
        ctypes.byref(cfg), _ptr(packed), _ptr(k_cache), _ptr(v_cache), int(cap), int(prefix_len),
        tok_p, par_p, int(n), _ptr(logits), _ptr(path), _ptr(accept_len), _ptr(next_token),
        _ptr(workspace), workspace.numel() * workspace.element_size(), _stream(stream))
    if raise_on_error:
        _check(rc, "llmcad_verify_tree")
    return rc


SCRATCH_BYTES = 96 << 20  # LLMCAD_SCRATCH_BYTES


def verify_tree_noalloc(cfg, packed, k_cache, v_cache, prefix_len: int, tree_tokens, parent, logits, path,
                        accept_len, next_token, status=None, stream=None, raise_on_error=True) -> int:
    """Enqueue one verification pass on the library's own scratch buffer (no
    workspace argument, no allocation); `status` (device int32 [1] or None)
    receives the pass's device status."""
    tok, tok_p = _i32(tree_tokens)
    par, par_p = _i32(parent)
    n = len(tok)
    if len(par) != n:
        raise ValueError("tree_tokens and parent differ in length")
    cap = k_cache.shape[-2]
    rc = _lib.llmcad_verify_tree_noalloc(
        ctypes.byref(cfg), _ptr(packed), _ptr(k_cache), _ptr(v_cache), int(cap), int(prefix_len),
        tok_p, par_p, int(n), _ptr(logits), _ptr(path), _ptr(accept_len), _ptr(next_token), _ptr(status),
        _stream(stream))
    if raise_on_error:
        _check(rc, "llmcad_verify_tree_noalloc")
    return rc


def prefill(cfg, packed, k_cache, v_cache, tokens, start_pos: int, last_logits, workspace,
            stream=None, raise_on_error=True) -> int:
    tok, tok_p = _i32(tokens)
    cap = k_cache.shape[-2]
    rc = _lib.llmcad_prefill(
        ctypes.byref(cfg), _ptr(packed), _ptr(k_cache), _ptr(v_cache), int(cap), tok_p, int(len(tok)),
        int(start_pos), _ptr(last_logits), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream))
    if raise_on_error:
        _check(rc, "llmcad_prefill")
    return rc


def extend_tree(cfg, packed, k_cache, v_cache, prefix_len: int, tree_tokens, parent, first: int, logits,
                workspace, stream=None, raise_on_error=True) -> int:
    """Tree-decoder step: the forward of nodes [first, n) of the tree (see llmcad_extend_tree)."""
    tok, tok_p = _i32(tree_tokens)
    par, par_p = _i32(parent)
    if len(par) != len(tok):
        raise ValueError("tree_tokens and parent differ in length")
    cap = k_cache.shape[-2]
    rc = _lib.llmcad_extend_tree(
        ctypes.byref(cfg), _ptr(packed), _ptr(k_cache), _ptr(v_cache), int(cap), int(prefix_len), tok_p, par_p,
        int(len(tok)), int(first), _ptr(logits), _ptr(workspace), workspace.numel() * workspace.element_size(),
        _stream(stream))
    if raise_on_error:
        _check(rc, "llmcad_extend_tree")
    return rc


CAND_MAX = 64  # LLMCAD_CAND_MAX
CAND_WORDS = 4 + 2 * CAND_MAX  # int32 words of one llmcad_candidates record


def extend_tree_candidates(cfg, packed, k_cache, v_cache, prefix_len: int, tree_tokens, parent, first: int,
                           threshold: float, logits, cand, workspace, stream=None, raise_on_error=True) -> int:
    """Tree-decoder step with candidate summaries (see llmcad_extend_tree_candidates):
    cand is a device int32 tensor of at least (n - first) x CAND_WORDS words."""
    tok, tok_p = _i32(tree_tokens)
    par, par_p = _i32(parent)
    if len(par) != len(tok):
        raise ValueError("tree_tokens and parent differ in length")
    if cand.dtype != torch.int32 or cand.numel() < (len(tok) - first) * CAND_WORDS:
        raise ValueError("cand must be an int32 device tensor of (n - first) records")
    cap = k_cache.shape[-2]
    rc = _lib.llmcad_extend_tree_candidates(
        ctypes.byref(cfg), _ptr(packed), _ptr(k_cache), _ptr(v_cache), int(cap), int(prefix_len), tok_p, par_p,
        int(len(tok)), int(first), float(threshold), _ptr(logits), _ptr(cand), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream))
    if raise_on_error:
        _check(rc, "llmcad_extend_tree_candidates")
    return rc


def parse_candidates(words):
    """One llmcad_candidates record (int32 numpy array of CAND_WORDS words) ->
    dict(count, argmax, max_logit, sum_exp, tok (list), prob (list))."""
    w = np.asarray(words, dtype=np.int32)
    f = w.view(np.float32)
    count = int(w[0])
    k = max(count, 0)
    return {"count": count, "argmax": int(w[1]), "max_logit": float(f[2]), "sum_exp": float(f[3]),
            "tok": [int(x) for x in w[4:4 + k]], "prob": [float(x) for x in f[4 + CAND_MAX:4 + CAND_MAX + k]]}


def commit_path(cfg, k_cache, v_cache, prefix_len: int, path, accept_len, n: int, stream=None,
                raise_on_error=True) -> int:
    """Rollback to the verified sequence: path/accept_len are the device outputs of the
    verification pass over n nodes at prefix_len (see llmcad_commit_path)."""
    cap = k_cache.shape[-2]
    rc = _lib.llmcad_commit_path(ctypes.byref(cfg), _ptr(k_cache), _ptr(v_cache), int(cap), int(prefix_len),
                                 _ptr(path), _ptr(accept_len), int(n), _stream(stream))
    if raise_on_error:
        _check(rc, "llmcad_commit_path")
    return rc


def workspace_region(cfg, n: int, which: int):
    off, size = ctypes.c_size_t(), ctypes.c_size_t()
    _check(_lib.llmcad_workspace_region(ctypes.byref(cfg), int(n), int(which), ctypes.byref(off),
                                        ctypes.byref(size)), "llmcad_workspace_region")
    return off.value, size.value


def timing_enable(kernel_class: int, max_launches: int):
    _check(_lib.llmcad_timing_enable(int(kernel_class), int(max_launches)), "llmcad_timing_enable")


def timing_read(kernel_class: int):
    """(summed milliseconds, launches) of the bracketed launches since the last read."""
    ms, n = ctypes.c_double(), ctypes.c_int32()
    _check(_lib.llmcad_timing_read(int(kernel_class), ctypes.byref(ms), ctypes.byref(n)),
           "llmcad_timing_read")
    return ms.value, n.value


class Session:
    """Owns the device buffers of one target model: packed weights, KV cache,
    workspace and output buffers (all torch tensors), and forwards calls."""

    def __init__(self, shape, capacity: int, max_n: int = MAX_NODES, device="cuda"):
        self.cfg = make_config(shape)
        rc = check_config(self.cfg)
        if rc != OK:
            raise LlmcadError(rc, "config")
        self.shape = shape
        self.device = torch.device(device)
        self.max_n = int(max_n)
        self.capacity = (int(capacity) + 63) // 64 * 64  # (the library takes multiples of 64)
        cap = self.capacity
        L, H, Dh = shape.n_layers, shape.n_heads, shape.head_dim
        self.packed = torch.empty(packed_bytes(self.cfg), dtype=torch.uint8, device=self.device)
        # K [L][H][cap][Dh]; V transposed per head [L][H][Dh][cap].  v_rows is
        # a [L][H][cap][Dh] view of the V cache (slot-major, like k_cache).
        self.k_cache = torch.zeros((L, H, cap, Dh), dtype=torch.bfloat16, device=self.device)
        self.v_cache = torch.zeros((L, H, Dh, cap), dtype=torch.bfloat16, device=self.device)
        self.v_rows = self.v_cache.transpose(2, 3)
        self.workspace = torch.zeros(workspace_bytes(self.cfg, self.max_n), dtype=torch.uint8,
                                     device=self.device)
        self.logits = torch.empty((self.max_n, shape.vocab), dtype=torch.float32, device=self.device)
        self.path = torch.empty(self.max_n, dtype=torch.int32, device=self.device)
        self.accept_len = torch.empty(1, dtype=torch.int32, device=self.device)
        self.next_token = torch.empty(1, dtype=torch.int32, device=self.device)
        self.last_logits = torch.empty(shape.vocab, dtype=torch.float32, device=self.device)
        off, _ = workspace_region(self.cfg, self.max_n, 5)  # (same offset for every pass size)
        self._status = self.workspace[off:off + 4].view(torch.int32)
        self._status_host = torch.zeros(1, dtype=torch.int32, pin_memory=True)

    def pass_status(self) -> int:
        """The device status of the passes enqueued so far (synchronises the stream)."""
        self._status_host.copy_(self._status, non_blocking=True)
        torch.cuda.current_stream().synchronize()
        return int(self._status_host[0])

    def check(self, what="pass"):
        """Raise LlmcadPassError if a pass since the last check failed on the device.
        The workspace's counters and status are cleared first, so the session
        serves the next pass; the failed pass's outputs (and the tree K/V it
        wrote) are invalid."""
        st = self.pass_status()
        if st != PASS_OK:
            workspace_init(self.cfg, self.max_n, self.workspace)
            torch.cuda.current_stream().synchronize()
            raise LlmcadPassError(st, what)

    def load_weights(self, gen, layers=None):
        """Pack weights from a generator with tok_embed(), final_norm(), lm_head(), layer(l)
        returning plain-layout tensors on this device (bf16 matrices, or for a
        4-bit model (codes, scales) pairs as pack_layer_q4 takes them)."""
        pack_globals(self.cfg, gen.tok_embed(), gen.final_norm(), gen.lm_head(), self.packed)
        q4 = self.cfg.weight_bits == 4
        for l in range(self.shape.n_layers) if layers is None else layers:
            (pack_layer_q4 if q4 else pack_layer)(self.cfg, l, gen.layer(l), self.packed)
            torch.cuda.current_stream().synchronize()  # let the plain layer be freed

    def prefill(self, tokens, start_pos=0, want_logits=False):
        prefill(self.cfg, self.packed, self.k_cache, self.v_cache, tokens, start_pos,
                self.last_logits if want_logits else None, self.workspace)
        return self.last_logits if want_logits else None

    def verify_tree(self, prefix_len, tree_tokens, parent, want_logits=True):
        n = len(tree_tokens)
        verify_tree(self.cfg, self.packed, self.k_cache, self.v_cache, prefix_len, tree_tokens,
                    parent, self.logits if want_logits else None, self.path, self.accept_len,
                    self.next_token, self.workspace)
        return n

    def extend(self, prefix_len, tree_tokens, parent, first):
        """Forward of nodes [first, n) of the tree; returns their logits [n - first, V] (device)."""
        n = len(tree_tokens)
        extend_tree(self.cfg, self.packed, self.k_cache, self.v_cache, prefix_len, tree_tokens, parent, first,
                    self.logits, self.workspace)
        return self.logits[: n - first]

    def extend_candidates(self, prefix_len, tree_tokens, parent, first, threshold):
        """Forward of nodes [first, n) with candidate summaries; returns one parsed
        record per computed row (synchronises; checks the device status)."""
        rows = len(tree_tokens) - first
        if not hasattr(self, "_cand"):
            self._cand = torch.zeros((self.max_n, CAND_WORDS), dtype=torch.int32, device=self.device)
            self._cand_host = torch.zeros((self.max_n, CAND_WORDS), dtype=torch.int32, pin_memory=True)
        extend_tree_candidates(self.cfg, self.packed, self.k_cache, self.v_cache, prefix_len, tree_tokens, parent,
                               first, threshold, self.logits, self._cand, self.workspace)
        h = self._cand_host
        h[:rows].copy_(self._cand[:rows], non_blocking=True)
        self.check("tree-decoder step")
        return [parse_candidates(h[i].numpy()) for i in range(rows)]

    def commit(self, prefix_len, n):
        """Roll the cache back to the verified sequence of the last verify_tree over n nodes."""
        commit_path(self.cfg, self.k_cache, self.v_cache, prefix_len, self.path, self.accept_len, n)

    def outcome(self):
        """After verify_tree: synchronise, check the device status, and return
        (path list, accept_len, next_token) -- four small copies, one sync."""
        if not hasattr(self, "_out_host"):
            self._out_host = torch.zeros(self.max_n + 3, dtype=torch.int32, pin_memory=True)
        h = self._out_host
        h[0:1].copy_(self._status, non_blocking=True)
        h[1:2].copy_(self.accept_len, non_blocking=True)
        h[2:3].copy_(self.next_token, non_blocking=True)
        h[3:].copy_(self.path, non_blocking=True)
        torch.cuda.current_stream().synchronize()
        st = int(h[0])
        if st != PASS_OK:
            workspace_init(self.cfg, self.max_n, self.workspace)
            torch.cuda.current_stream().synchronize()
            raise LlmcadPassError(st, "verification pass")
        acc = int(h[1])
        return [int(x) for x in h[3:3 + acc + 1]], acc, int(h[2])

    def results(self, n):
        """Synchronise, check the device status, and return (logits [n, V] fp32 cpu,
        path list, accept_len, next_token)."""
        self.check("verification pass")
        acc = int(self.accept_len.item())
        return (self.logits[:n].cpu(), [int(x) for x in self.path[: acc + 1].cpu()], acc,
                int(self.next_token.item()))
