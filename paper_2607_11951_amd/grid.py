"""Thin Python binding of libgrid.so (the C ABI in include/grid.h).

Argument marshalling only: every step of the mask path runs in the library's
HIP kernels.  PyTorch provides device memory and the stream.  The binding
refuses to run when the library is missing -- there is no fallback.
"""

import ctypes
from pathlib import Path

import numpy as np

PKG = Path(__file__).resolve().parent
LIB_PATH = PKG / "libgrid.so"

GRID_OK = 0
ERRORS = {
    -1: "GRID_E_ARG", -2: "GRID_E_GRAMMAR_SYNTAX", -3: "GRID_E_LALR_CONFLICT",
    -4: "GRID_E_EMPTY_LANGUAGE", -5: "GRID_E_LEXICON", -6: "GRID_E_LEXER_GAP",
    -7: "GRID_E_VOCAB", -8: "GRID_E_NOT_VIABLE", -9: "GRID_E_UNBOUND", -10: "GRID_E_HIP",
    -11: "GRID_E_CAPACITY",
}
ROW_OK, ROW_EMPTY, ROW_BAD_CONFIG, ROW_OVERFLOW, ROW_NOT_VIABLE, ROW_FINISHED = 0, 1, 2, 4, 8, 16
CACHE_LOOKUP, CACHE_INSERT = 1, 2
DTYPE_F32, DTYPE_BF16 = 0, 1

ART_NAMES = ["DFA_DENSE", "DFA_CLASS", "BYTE_CLASS", "DFA_ACCEPT_OFF", "DFA_ACCEPT_LIST", "DFA_LIVE",
             "ACTION", "GOTO", "PROD", "TERM_INFO", "SPELL_OFF", "SPELL_BYTES", "ALIAS_OFF",
             "ALIAS_IDS", "TRIE_LEVEL_OFF", "TRIE_NODES", "LEX_FLAGS", "LEX_HASH", "LEX_SLOTS",
             "SPELL_REC", "PARSE_STATE", "PARSE_REDX", "GOTO_HASH", "SPELL_TAIL", "LEX_PREFIX",
             "SPELL_RANGE", "SPELL_OF_ID", "CLASS_MAP", "CLASS_OFF", "CLASS_REC", "LEX_STRIDE",
             "LEX_TOKEN", "ID_FIRST", "PARSE_SHIFT", "STATE_SYMBOL", "LEX_CHILD", "ID_HEAD",
             "LEX_TOKSUM", "GOTO_SKIP"]
ART = {n: i for i, n in enumerate(ART_NAMES)}

CONFIG_DTYPE = np.dtype([("stk_off", "<u4"), ("stk_depth", "<u4"), ("lexnode", "<u4"), ("q", "<u2"),
                         ("slot", "<u2"), ("flags", "<u4"), ("rem_len", "<u4"),
                         ("rem_head", "u1", (8,))])
assert CONFIG_DTYPE.itemsize == 32

# every symbol include/grid.h declares
EXPORTS = ["grid_compile", "grid_free", "grid_last_error", "grid_info", "grid_add_lexicon",
           "grid_artifact", "grid_bind_device", "grid_config_from_prefix",
           "grid_mask_workspace_bytes", "grid_mask", "grid_mask_phases", "grid_apply",
           "grid_cache_bytes", "grid_cache_clear", "grid_mask_cached", "grid_accept",
           "grid_mask_noalloc_max_bytes", "grid_mask_noalloc", "grid_stack_hash", "grid_stack_hash_host",
           "grid_accept_inplace", "grid_ci_cache_bytes", "grid_ci_cache_clear", "grid_mask_warm",
           "grid_complete", "grid_forced_span", "grid_forced_span_workspace_bytes"]
CI_LOOKUP, CI_INSERT, CI_FAMILY, CI_GENN = 1, 2, 4, 8
PHASE_PROLOGUE, PHASE_WALK, PHASE_RESIDUE, PHASE_FINALIZE, PHASE_ALL = 1, 2, 4, 8, 15


class GridError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


class _CompileArgs(ctypes.Structure):
    _fields_ = [("grammar", ctypes.c_char_p), ("grammar_len", ctypes.c_size_t),
                ("drop_labels", ctypes.c_char_p), ("vocab_bytes", ctypes.c_void_p),
                ("vocab_offsets", ctypes.c_void_p), ("vocab_size", ctypes.c_int32),
                ("special_ids", ctypes.c_void_p), ("n_special", ctypes.c_int32),
                ("eos_id", ctypes.c_int32)]


class _LexiconArgs(ctypes.Structure):
    _fields_ = [("n_categories", ctypes.c_int32), ("names", ctypes.POINTER(ctypes.c_char_p)),
                ("words", ctypes.POINTER(ctypes.c_char_p))]


class _Info(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_terminals", "n_nonterminals", "n_productions", "n_lr_states", "n_dfa_states",
        "n_byte_classes", "vocab_size", "mask_words", "n_spellings", "max_spelling_len",
        "n_trie_nodes", "n_lexicon_slots", "byte_complete", "overlay_capacity")]


_lib = None


def lib():
    """The loaded library; raises if it was not built."""
    global _lib
    if _lib is None:
        if not LIB_PATH.exists():
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(str(LIB_PATH))
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        L.grid_compile.argtypes = [ctypes.POINTER(_CompileArgs), ctypes.POINTER(vp)]
        L.grid_free.argtypes = [vp]
        L.grid_free.restype = None
        L.grid_last_error.restype = ctypes.c_char_p
        L.grid_info.argtypes = [vp, ctypes.POINTER(_Info)]
        L.grid_add_lexicon.argtypes = [vp, ctypes.POINTER(_LexiconArgs), ctypes.POINTER(i32)]
        L.grid_artifact.argtypes = [vp, i32, ctypes.POINTER(vp), ctypes.POINTER(sz)]
        L.grid_bind_device.argtypes = [vp, i32, vp]
        L.grid_config_from_prefix.argtypes = [vp, i32, ctypes.c_char_p, sz, vp, vp, ctypes.c_uint32,
                                              ctypes.POINTER(ctypes.c_uint32)]
        L.grid_mask_workspace_bytes.argtypes = [vp, i32]
        L.grid_mask_workspace_bytes.restype = sz
        L.grid_mask.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp, sz, vp]
        L.grid_mask_phases.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp, sz, ctypes.c_uint32, vp]
        L.grid_apply.argtypes = [vp, vp, i32, i32, i32, ctypes.c_int64, vp]
        L.grid_accept.argtypes = [vp, i32, vp, vp, vp, vp, vp, ctypes.c_uint32, vp, vp]
        L.grid_mask_cached.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp, sz, ctypes.c_uint32, vp]
        L.grid_stack_hash.argtypes = [vp, i32, vp, vp, vp, vp]
        L.grid_stack_hash_host.argtypes = [vp, vp, ctypes.c_uint32, vp]
        L.grid_accept_inplace.argtypes = [vp, i32, vp, vp, vp, ctypes.c_uint32, vp, vp, vp]
        L.grid_complete.argtypes = [vp, i32, ctypes.c_char_p, sz, i32, vp, ctypes.POINTER(i32)]
        L.grid_forced_span.argtypes = [vp, i32, vp, vp, vp, ctypes.c_uint32, i32, vp, vp, vp, vp, vp, vp, sz, vp]
        L.grid_forced_span_workspace_bytes.argtypes = [vp, i32]
        L.grid_forced_span_workspace_bytes.restype = sz
        L.grid_ci_cache_bytes.argtypes = [vp, i32]
        L.grid_ci_cache_bytes.restype = sz
        L.grid_ci_cache_clear.argtypes = [vp, vp, sz, vp]
        L.grid_mask_warm.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp, sz, vp, sz, ctypes.c_uint32, vp]
        L.grid_cache_bytes.argtypes = [vp, i32]
        L.grid_cache_bytes.restype = sz
        L.grid_cache_clear.argtypes = [vp, vp, sz, vp]
        L.grid_mask_noalloc_max_bytes.argtypes = []
        L.grid_mask_noalloc_max_bytes.restype = sz
        L.grid_mask_noalloc.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp]
        _lib = L
    return _lib


def _check(rc):
    if rc != GRID_OK:
        raise GridError(rc, lib().grid_last_error().decode(errors="replace"))


def _stream_handle(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


class Grid:
    """A compiled grammar + role projection + vocabulary, plus lexicon slots."""

    def __init__(self, grammar_text, drop=(), vocab=(), specials=(), eos_id=-1):
        vocab = list(vocab)
        offs = np.zeros(len(vocab) + 1, dtype=np.uint64)
        offs[1:] = np.cumsum([len(t) for t in vocab], dtype=np.uint64)
        data = np.frombuffer(b"".join(vocab) + b"\0", dtype=np.uint8)
        sp = np.asarray(list(specials) or [0], dtype=np.int32)
        text = grammar_text.encode()
        drop_s = ",".join(drop).encode() if drop else None
        args = _CompileArgs(text, len(text), drop_s, data.ctypes.data, offs.ctypes.data, len(vocab),
                            sp.ctypes.data, len(specials), eos_id)
        h = ctypes.c_void_p()
        _check(lib().grid_compile(ctypes.byref(args), ctypes.byref(h)))
        self._lib_ref = lib()  # kept so that the handle can be freed during interpreter shutdown
        self.h = h
        self.V = len(vocab)
        self.W = (self.V + 31) // 32
        self._dev = {}
        self.device = None

    def __del__(self):
        L = getattr(self, "_lib_ref", None)
        if getattr(self, "h", None) and L is not None:
            L.grid_free(self.h)
            self.h = None

    def info(self):
        inf = _Info()
        _check(lib().grid_info(self.h, ctypes.byref(inf)))
        return {n: getattr(inf, n) for n, _ in _Info._fields_}

    def add_lexicon(self, cats):
        names = list(cats)
        arr_n = (ctypes.c_char_p * max(1, len(names)))(*[n.encode() for n in names])
        arr_w = (ctypes.c_char_p * max(1, len(names)))(*["\n".join(cats[n]).encode() for n in names])
        la = _LexiconArgs(len(names), arr_n, arr_w)
        slot = ctypes.c_int32()
        _check(lib().grid_add_lexicon(self.h, ctypes.byref(la), ctypes.byref(slot)))
        if self.device is not None:
            self._upload(self.device, ["LEX_FLAGS", "LEX_HASH", "LEX_SLOTS", "LEX_PREFIX", "LEX_STRIDE", "LEX_TOKEN",
                                       "LEX_CHILD", "LEX_TOKSUM"])
        return slot.value

    def artifact(self, name):
        p, n = ctypes.c_void_p(), ctypes.c_size_t()
        _check(lib().grid_artifact(self.h, ART[name], ctypes.byref(p), ctypes.byref(n)))
        if n.value == 0:
            return b""
        return ctypes.string_at(p.value, n.value)

    def _upload(self, device, names):
        import torch
        for name in names:
            raw = self.artifact(name)
            if raw:
                t = torch.frombuffer(bytearray(raw), dtype=torch.uint8).to(device)
                ptr = t.data_ptr()
            else:
                t, ptr = None, None
            self._dev[name] = t
            _check(lib().grid_bind_device(self.h, ART[name], ctypes.c_void_p(ptr)))

    def to_device(self, device="cuda"):
        """Copies every artifact to device memory and binds it."""
        self.device = device
        self._upload(device, ART_NAMES)
        return self

    def config(self, w, slot=0, cap=1 << 16):
        """(grid_config record, stack states) for prefix bytes w; raises
        GridError(GRID_E_NOT_VIABLE) if w is not a viable prefix."""
        cfg = np.zeros(1, dtype=CONFIG_DTYPE)
        stack = np.zeros(cap, dtype=np.uint16)
        depth = ctypes.c_uint32()
        _check(lib().grid_config_from_prefix(self.h, slot, w, len(w), cfg.ctypes.data, stack.ctypes.data,
                                             cap, ctypes.byref(depth)))
        return cfg[0], stack[: depth.value].copy()

    def configs(self, prefixes, slots=None):
        """Host arrays (configs, stack pool) for a batch of prefixes."""
        if slots is None:
            slots = [0] * len(prefixes)
        cfgs = np.zeros(len(prefixes), dtype=CONFIG_DTYPE)
        pool = []
        off = 0
        for i, (w, s) in enumerate(zip(prefixes, slots)):
            c, st = self.config(w, s)
            c["stk_off"] = off
            cfgs[i] = c
            pool.append(st)
            off += len(st)
        return cfgs, np.concatenate(pool) if pool else np.zeros(1, np.uint16)

    def configs_to_device(self, cfgs, pool, device=None):
        import torch
        device = device or self.device
        c = torch.from_numpy(cfgs.view(np.uint8).copy()).to(device)
        p = torch.from_numpy(pool.view(np.int16).copy()).to(device)
        return c, p

    def accept(self, cfg_dev, pool_dev, tokens_dev, B, stack_cap, out=None, stack_out=None, status=None,
               stream=None):
        """Device incremental advance (grid_accept): row b's configuration followed by
        token tokens_dev[b].  Returns (configs uint8 [B * 32], stack pool int16
        [B * stack_cap], status int32 [B]); the first two are the next step's inputs."""
        import torch
        dev = cfg_dev.device
        if out is None:
            out = torch.empty(B * 32, dtype=torch.uint8, device=dev)
        if stack_out is None:
            stack_out = torch.empty(B * stack_cap, dtype=torch.int16, device=dev)
        if status is None:
            status = torch.empty(B, dtype=torch.int32, device=dev)
        assert tokens_dev.dtype == torch.int32 and tokens_dev.numel() >= B
        _check(lib().grid_accept(self.h, B, ctypes.c_void_p(cfg_dev.data_ptr()),
                                 ctypes.c_void_p(pool_dev.data_ptr()), ctypes.c_void_p(tokens_dev.data_ptr()),
                                 ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(stack_out.data_ptr()),
                                 stack_cap, ctypes.c_void_p(status.data_ptr()), _stream_handle(stream)))
        return out, stack_out, status

    def accept_inplace(self, cfg_dev, pool_dev, tokens_dev, B, stack_cap, stack_hash=None, status=None,
                       stream=None):
        """grid_accept_inplace: row b's configuration cfg_dev[b] (stack at
        pool_dev[b * stack_cap ..]) advanced in place by tokens_dev[b]; the
        rolling hashes in stack_hash (uint64/int64 tensor parallel to the pool)
        are kept up to date.  Returns the status tensor."""
        import torch
        if status is None:
            status = torch.empty(B, dtype=torch.int32, device=cfg_dev.device)
        assert tokens_dev.dtype == torch.int32 and tokens_dev.numel() >= B
        assert pool_dev.numel() >= B * stack_cap
        hp = ctypes.c_void_p(stack_hash.data_ptr()) if stack_hash is not None else None
        _check(lib().grid_accept_inplace(self.h, B, ctypes.c_void_p(cfg_dev.data_ptr()),
                                         ctypes.c_void_p(pool_dev.data_ptr()), hp, stack_cap,
                                         ctypes.c_void_p(tokens_dev.data_ptr()), ctypes.c_void_p(status.data_ptr()),
                                         _stream_handle(stream)))
        return status

    def forced_span(self, cfg_dev, pool_dev, B, stack_cap, max_len, stack_hash=None, workspace=None,
                    stream=None):
        """grid_forced_span: rows advanced in place by their forced spans (at
        most max_len tokens).  Returns (span int32 [B, max_len] with -1 after
        each row's span, span_len int32 [B], and the mask, eos and status of
        the final configurations)."""
        import torch
        dev = cfg_dev.device
        assert pool_dev.numel() >= B * stack_cap and max_len >= 1
        span = torch.empty((B, max_len), dtype=torch.int32, device=dev)
        span_len = torch.empty(B, dtype=torch.int32, device=dev)
        out = torch.empty((B, self.W), dtype=torch.int32, device=dev)
        eos = torch.empty(B, dtype=torch.uint8, device=dev)
        status = torch.empty(B, dtype=torch.int32, device=dev)
        if workspace is None:
            workspace = torch.empty(lib().grid_forced_span_workspace_bytes(self.h, B), dtype=torch.uint8, device=dev)
        hp = ctypes.c_void_p(stack_hash.data_ptr()) if stack_hash is not None else None
        _check(lib().grid_forced_span(self.h, B, ctypes.c_void_p(cfg_dev.data_ptr()),
                                      ctypes.c_void_p(pool_dev.data_ptr()), hp, stack_cap, max_len,
                                      ctypes.c_void_p(span.data_ptr()), ctypes.c_void_p(span_len.data_ptr()),
                                      ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(eos.data_ptr()),
                                      ctypes.c_void_p(status.data_ptr()), ctypes.c_void_p(workspace.data_ptr()),
                                      workspace.numel(), _stream_handle(stream)))
        return span, span_len, out, eos, status

    def stack_hash(self, cfg_dev, pool_dev, B, out=None, stream=None):
        """grid_stack_hash: the rolling hash of every pool entry of the B rows'
        stacks (int64 tensor parallel to the pool; entries outside the rows'
        stacks are left as they are)."""
        import torch
        if out is None:
            out = torch.zeros(pool_dev.numel(), dtype=torch.int64, device=pool_dev.device)
        _check(lib().grid_stack_hash(self.h, B, ctypes.c_void_p(cfg_dev.data_ptr()),
                                     ctypes.c_void_p(pool_dev.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                                     _stream_handle(stream)))
        return out

    def complete(self, w, slot=0, max_tokens=4096):
        """grid_complete: token ids of a legal completion of the viable prefix w
        (their number is w's reserve)."""
        out = np.zeros(max(1, max_tokens), dtype=np.int32)
        n = ctypes.c_int32()
        _check(lib().grid_complete(self.h, slot, w, len(w), max_tokens, out.ctypes.data, ctypes.byref(n)))
        return out[:n.value].copy()

    def stack_hash_host(self, states):
        """grid_stack_hash_host: the rolling hashes of one stack (uint64 array)."""
        st = np.ascontiguousarray(states, dtype=np.uint16)
        out = np.zeros(len(st), dtype=np.uint64)
        _check(lib().grid_stack_hash_host(self.h, st.ctypes.data, len(st), out.ctypes.data))
        return out

    def workspace_bytes(self, B):
        return lib().grid_mask_workspace_bytes(self.h, B)

    def new_workspace(self, B, device=None):
        import torch
        return torch.empty(self.workspace_bytes(B), dtype=torch.uint8, device=device or self.device)

    def cache_bytes(self, n_entries):
        """Device bytes of a mask cache of n_entries (a power of two) entries."""
        n = lib().grid_cache_bytes(self.h, n_entries)
        if n == 0:
            raise ValueError("n_entries must be a power of two")
        return n

    def new_cache(self, n_entries, device=None, stream=None):
        """A cleared mask cache (uint8 device tensor)."""
        import torch
        c = torch.empty(self.cache_bytes(n_entries), dtype=torch.uint8, device=device or self.device)
        self.clear_cache(c, stream)
        return c

    def new_ci_cache(self, n_entries, device=None, stream=None):
        """A cleared cache of context-independent words (uint8 device tensor)."""
        import torch
        n = lib().grid_ci_cache_bytes(self.h, n_entries)
        if n == 0:
            raise ValueError("n_entries must be a power of two")
        c = torch.empty(n, dtype=torch.uint8, device=device or self.device)
        _check(lib().grid_ci_cache_clear(self.h, ctypes.c_void_p(c.data_ptr()), c.numel(), _stream_handle(stream)))
        return c

    def clear_ci_cache(self, ci_cache, stream=None):
        _check(lib().grid_ci_cache_clear(self.h, ctypes.c_void_p(ci_cache.data_ptr()), ci_cache.numel(),
                                         _stream_handle(stream)))

    def mask_warm(self, cfg_dev, pool_dev, B, ci_cache, flags=1 | 2, out=None, eos=None, status=None,
                  workspace=None, stream=None):
        """grid_mask_warm: the mask of B rows with the CI-words cache (CI_* flags)."""
        import torch
        dev = cfg_dev.device
        if out is None:
            out = torch.empty((B, self.W), dtype=torch.int32, device=dev)
        if eos is None:
            eos = torch.empty(B, dtype=torch.uint8, device=dev)
        if status is None:
            status = torch.empty(B, dtype=torch.int32, device=dev)
        if workspace is None:
            workspace = self.new_workspace(B, dev)
        assert cfg_dev.numel() >= 32 * B and out.numel() >= B * self.W and out.is_contiguous()
        _check(lib().grid_mask_warm(self.h, B, ctypes.c_void_p(cfg_dev.data_ptr()),
                                    ctypes.c_void_p(pool_dev.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                                    ctypes.c_void_p(eos.data_ptr()), ctypes.c_void_p(status.data_ptr()),
                                    ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                                    ctypes.c_void_p(ci_cache.data_ptr()), ci_cache.numel(), flags,
                                    _stream_handle(stream)))
        return out, eos, status

    def clear_cache(self, cache, stream=None):
        _check(lib().grid_cache_clear(self.h, ctypes.c_void_p(cache.data_ptr()), cache.numel(),
                                      _stream_handle(stream)))

    def mask(self, cfg_dev, pool_dev, B, out=None, eos=None, status=None, workspace=None, stream=None,
             phases=PHASE_ALL, cache=None, cache_flags=CACHE_LOOKUP | CACHE_INSERT, stack_hash=None):
        """Enqueues the mask of B rows; returns (mask int32 [B, W], eos u8 [B], status i32 [B]).
        phases selects a subset of the launches (grid_mask_phases); cache (from new_cache)
        serves and records rows through the mask cache (grid_mask_cached), keyed by the
        rolling stack hashes stack_hash (from stack_hash) when given."""
        import torch
        dev = cfg_dev.device
        if out is None:
            out = torch.empty((B, self.W), dtype=torch.int32, device=dev)
        if eos is None:
            eos = torch.empty(B, dtype=torch.uint8, device=dev)
        if status is None:
            status = torch.empty(B, dtype=torch.int32, device=dev)
        if workspace is None:
            workspace = self.new_workspace(B, dev)
        assert cfg_dev.numel() >= 32 * B and out.numel() >= B * self.W and out.is_contiguous()
        head = (self.h, B, ctypes.c_void_p(cfg_dev.data_ptr()), ctypes.c_void_p(pool_dev.data_ptr()))
        tail = (ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(eos.data_ptr()),
                ctypes.c_void_p(status.data_ptr()), ctypes.c_void_p(workspace.data_ptr()), workspace.numel())
        args = head + tail
        if cache is not None:
            assert phases == PHASE_ALL
            hp = ctypes.c_void_p(stack_hash.data_ptr()) if stack_hash is not None else None
            _check(lib().grid_mask_cached(*head, hp, *tail, ctypes.c_void_p(cache.data_ptr()), cache.numel(),
                                          cache_flags, _stream_handle(stream)))
        elif phases == PHASE_ALL:
            _check(lib().grid_mask(*args, _stream_handle(stream)))
        else:
            _check(lib().grid_mask_phases(*args, phases, _stream_handle(stream)))
        return out, eos, status


def mask_noalloc(grid, cfg_dev, pool_dev, B, out, eos, status, stream=None):
    """grid_mask_noalloc: the mask of B rows into caller tensors, with the
    library's static device scratch as workspace (nothing is allocated)."""
    assert cfg_dev.numel() >= 32 * B and out.numel() >= B * grid.W and out.is_contiguous()
    assert eos.numel() >= B and status.numel() >= B
    _check(lib().grid_mask_noalloc(grid.h, B, ctypes.c_void_p(cfg_dev.data_ptr()),
                                   ctypes.c_void_p(pool_dev.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                                   ctypes.c_void_p(eos.data_ptr()), ctypes.c_void_p(status.data_ptr()),
                                   _stream_handle(stream)))
    return out, eos, status


def apply(mask, logits, stream=None):
    """In-place -inf fill of logits [B, V] (fp32 or bf16) where the mask bit is 0."""
    import torch
    B, V = logits.shape
    if logits.dtype == torch.bfloat16:
        dt = DTYPE_BF16
    elif logits.dtype == torch.float32:
        dt = DTYPE_F32
    else:
        raise TypeError("logits must be float32 or bfloat16")
    assert logits.stride(1) == 1 and mask.shape[0] == B and mask.shape[1] >= (V + 31) // 32
    _check(lib().grid_apply(ctypes.c_void_p(mask.data_ptr()), ctypes.c_void_p(logits.data_ptr()), dt, B, V,
                            logits.stride(0), _stream_handle(stream)))
    return logits


def from_workload(wl):
    """A Grid for a workload (see the workloads package), with its lexicon slots."""
    from workloads import grammar_text
    g = Grid(grammar_text(wl.grammar), wl.drop, wl.vocab, wl.specials, wl.eos_id)
    slots = []
    for lex in wl.lexicons:
        slots.append(g.add_lexicon(lex) if lex else 0)
    return g, slots
