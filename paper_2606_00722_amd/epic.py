"""Python binding of the C ABI in include/epic.h (argument marshalling only).

Device buffers are PyTorch tensors on a HIP device; every call enqueues on the
given torch stream (default: the current stream).  All computation happens in
the HIP kernels of libepic.so; there is no fallback: if the library is not
built, loading it raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# EPIC_LIB names another build of the same library (e.g. a profiling build)
LIB_PATH = os.environ.get("EPIC_LIB") or os.path.join(HERE, "libepic.so")

STATUS = {0: "ok", -1: "null pointer", -2: "argument out of range", -3: "capacity exceeded",
          -4: "malformed lexer DFA", -5: "malformed grammar", -6: "malformed vocabulary",
          -7: "HIP runtime error", -8: "memo not built", -9: "unsupported size"}
DEV_BAD_CANDIDATE, DEV_CAPACITY, DEV_BAD_SELECT = 1, 2, 4

FUNCTIONS = ["epic_ctx_create", "epic_ctx_destroy", "epic_workspace_bytes", "epic_gap_classes", "epic_item_words",
             "epic_lexmemo_build", "epic_memo_export", "epic_validate_batch", "epic_validate_batch_noalloc",
             "epic_select_compatible",
             "epic_commit_fallback",
             "epic_ctx_device_error", "epic_ctx_work_counters", "epic_ctx_set_timing",
             "epic_ctx_set_witness_lds", "epic_ctx_kernel_stats",
             "epic_witness_workspace_bytes", "epic_witness",
             "epic_diag_lds_stream", "epic_diag_clock_rates", "epic_status_string"]
KERNEL_KINDS = ["lexmemo", "base", "validate", "select", "fallback", "spec_bookkeeping", "spec_unused"]


class EpicError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn}: {STATUS.get(code, code)} ({code})")
        self.code = code


class _Lexer(ctypes.Structure):
    _fields_ = [("num_states", ctypes.c_int32), ("trans", ctypes.c_void_p), ("accept", ctypes.c_void_p)]


class _Grammar(ctypes.Structure):
    _fields_ = [("num_terminals", ctypes.c_int32), ("num_nonterminals", ctypes.c_int32),
                ("start", ctypes.c_int32), ("num_productions", ctypes.c_int32),
                ("lhs", ctypes.c_void_p), ("rhs_offsets", ctypes.c_void_p), ("rhs", ctypes.c_void_p)]


class _Vocab(ctypes.Structure):
    _fields_ = [("vocab_size", ctypes.c_int32), ("bytes", ctypes.c_void_p), ("offsets", ctypes.c_void_p)]


_lib: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libepic.so is not built ({LIB_PATH}); run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        P, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        L.epic_ctx_create.argtypes = [P, P, P, i32, i32, i32, ctypes.POINTER(P)]
        L.epic_ctx_create.restype = ctypes.c_int
        L.epic_ctx_destroy.argtypes = [P]
        L.epic_ctx_destroy.restype = None
        L.epic_workspace_bytes.argtypes = [P]
        L.epic_workspace_bytes.restype = sz
        L.epic_gap_classes.argtypes = [P]
        L.epic_gap_classes.restype = i32
        L.epic_item_words.argtypes = [P]
        L.epic_item_words.restype = i32
        L.epic_lexmemo_build.argtypes = [P, P]
        L.epic_lexmemo_build.restype = ctypes.c_int
        L.epic_memo_export.argtypes = [P, P, sz]
        L.epic_memo_export.restype = ctypes.c_int
        L.epic_validate_batch.argtypes = [P, P, i32, i32, P, P, P, i32, P, P, sz, P]
        L.epic_validate_batch.restype = ctypes.c_int
        L.epic_validate_batch_noalloc.argtypes = [P, P, i32, i32, P, P, P, i32, P, P]
        L.epic_validate_batch_noalloc.restype = ctypes.c_int
        L.epic_select_compatible.argtypes = [P, P, i32, i32, P, P, P, P, P, i32, P, P, P, sz, P]
        L.epic_select_compatible.restype = ctypes.c_int
        L.epic_commit_fallback.argtypes = [P, P, i32, i32, P, P, P, P, P, P, P, i32, P, P, sz, P]
        L.epic_commit_fallback.restype = ctypes.c_int
        L.epic_ctx_device_error.argtypes = [P, P, ctypes.POINTER(ctypes.c_uint32)]
        L.epic_ctx_device_error.restype = ctypes.c_int
        L.epic_ctx_work_counters.argtypes = [P, P, P]
        L.epic_ctx_work_counters.restype = ctypes.c_int
        L.epic_ctx_set_timing.argtypes = [P, i32]
        L.epic_ctx_set_timing.restype = ctypes.c_int
        L.epic_ctx_set_witness_lds.argtypes = [P, i32, i32]
        L.epic_ctx_set_witness_lds.restype = ctypes.c_int
        L.epic_ctx_kernel_stats.argtypes = [P, P, P, P, P]
        L.epic_ctx_kernel_stats.restype = ctypes.c_int
        L.epic_witness_workspace_bytes.argtypes = [P, i32]
        L.epic_witness_workspace_bytes.restype = sz
        L.epic_witness.argtypes = [P, P, i32, i32, P, i32, P, i32, P, P, sz, P, sz, P]
        L.epic_witness.restype = ctypes.c_int
        L.epic_diag_lds_stream.argtypes = [i32, i32, i32, P, P]
        L.epic_diag_lds_stream.restype = ctypes.c_int
        L.epic_diag_clock_rates.argtypes = [ctypes.POINTER(i32), ctypes.POINTER(i32)]
        L.epic_diag_clock_rates.restype = ctypes.c_int
        L.epic_status_string.argtypes = [ctypes.c_int]
        L.epic_status_string.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(fn: str, code: int):
    if code != 0:
        raise EpicError(fn, code)


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _stream(stream) -> int:
    import torch

    s = torch.cuda.current_stream() if stream is None else stream
    return int(s.cuda_stream)


class Context:
    """An epic_ctx: lexer DFA, grammar and vocabulary tables on the device."""

    def __init__(self, trans, accept, num_terminals, num_nonterminals, start, lhs, rhs_offsets, rhs,
                 vocab_bytes, vocab_offsets, max_batch, max_seq_len, max_cands):
        self._keep = [np.ascontiguousarray(trans, np.int16), np.ascontiguousarray(accept, np.int16),
                      np.ascontiguousarray(lhs, np.int32), np.ascontiguousarray(rhs_offsets, np.int32),
                      np.ascontiguousarray(rhs if len(rhs) else np.zeros(1), np.int32),
                      np.ascontiguousarray(vocab_bytes if len(vocab_bytes) else np.zeros(1), np.uint8),
                      np.ascontiguousarray(vocab_offsets, np.int32)]
        tr, ac, lh, ro, rh, vb, vo = self._keep
        self.num_states = int(tr.shape[0])
        self.vocab_size = int(vo.shape[0] - 1)
        lx = _Lexer(self.num_states, tr.ctypes.data, ac.ctypes.data)
        gr = _Grammar(num_terminals, num_nonterminals, start, int(lh.shape[0]), lh.ctypes.data, ro.ctypes.data,
                      rh.ctypes.data)
        vc = _Vocab(self.vocab_size, vb.ctypes.data, vo.ctypes.data)
        h = ctypes.c_void_p()
        _check("epic_ctx_create", lib().epic_ctx_create(ctypes.byref(lx), ctypes.byref(gr), ctypes.byref(vc),
                                                         max_batch, max_seq_len, max_cands, ctypes.byref(h)))
        self._h = h

    @classmethod
    def from_problem(cls, p, max_batch, max_seq_len, max_cands):
        """From an object with the generator's arrays (trans, accept, T, N, start, lhs, roff, rhs, vbytes, voffs)."""
        return cls(p.trans, p.accept, p.T, p.N, p.start, p.lhs, p.roff, p.rhs, p.vbytes, p.voffs,
                   max_batch, max_seq_len, max_cands)

    def close(self):
        if getattr(self, "_h", None):
            lib().epic_ctx_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def workspace_bytes(self) -> int:
        return int(lib().epic_workspace_bytes(self._h))

    @property
    def gap_classes(self) -> int:
        return int(lib().epic_gap_classes(self._h))

    def alloc_workspace(self, device="cuda"):
        """A zeroed workspace (a fresh workspace must hold no walk records)."""
        import torch

        return torch.zeros(self.workspace_bytes + 256, dtype=torch.uint8, device=device)

    def alloc_witness_workspace(self, B: int, device="cuda"):
        """Device memory for epic_witness on B sequences (contents need not be cleared)."""
        import torch

        return torch.empty(self.witness_workspace_bytes(B) + 256, dtype=torch.uint8, device=device)

    def lexmemo_build(self, stream=None):
        _check("epic_lexmemo_build", lib().epic_lexmemo_build(self._h, _stream(stream)))

    def memo_export(self) -> np.ndarray:
        out = np.zeros((self.vocab_size, self.num_states, 16), dtype=np.uint8)
        _check("epic_memo_export", lib().epic_memo_export(self._h, out.ctypes.data, out.nbytes))
        return out

    @staticmethod
    def _ws(workspace):
        p = _ptr(workspace)
        aligned = (p + 255) & ~255
        return aligned, workspace.numel() - (aligned - p)

    def validate(self, seqs, cand_seq, cand_pos, cand_tok, verdict, workspace, stream=None):
        B, n = (int(seqs.shape[0]), int(seqs.shape[1])) if seqs.dim() == 2 else (0, 0)
        wp, wb = self._ws(workspace)
        _check("epic_validate_batch", lib().epic_validate_batch(
            self._h, _ptr(seqs), B, n, _ptr(cand_seq), _ptr(cand_pos), _ptr(cand_tok), int(cand_seq.numel()),
            _ptr(verdict), wp, wb, _stream(stream)))

    def validate_noalloc(self, seqs, cand_seq, cand_pos, cand_tok, verdict, stream=None):
        """epic_validate_batch_noalloc: no workspace (the library's static
        device scratch; calls on one GPU must not overlap)."""
        B, n = (int(seqs.shape[0]), int(seqs.shape[1])) if seqs.dim() == 2 else (0, 0)
        _check("epic_validate_batch_noalloc", lib().epic_validate_batch_noalloc(
            self._h, _ptr(seqs), B, n, _ptr(cand_seq), _ptr(cand_pos), _ptr(cand_tok), int(cand_seq.numel()),
            _ptr(verdict), _stream(stream)))

    def select(self, seqs, cand_seq, cand_pos, cand_tok, conf, verdict, selected, workspace, counts=None,
               stream=None):
        B, n = int(seqs.shape[0]), int(seqs.shape[1])
        wp, wb = self._ws(workspace)
        _check("epic_select_compatible", lib().epic_select_compatible(
            self._h, _ptr(seqs), B, n, _ptr(cand_seq), _ptr(cand_pos), _ptr(cand_tok), _ptr(conf), _ptr(verdict),
            int(cand_seq.numel()), _ptr(selected), _ptr(counts), wp, wb, _stream(stream)))

    def fallback(self, seqs, cand_seq, cand_pos, cand_tok, conf, verdict, selected, num_commit, accepted, workspace,
                 stream=None):
        B, n = int(seqs.shape[0]), int(seqs.shape[1])
        wp, wb = self._ws(workspace)
        _check("epic_commit_fallback", lib().epic_commit_fallback(
            self._h, _ptr(seqs), B, n, _ptr(cand_seq), _ptr(cand_pos), _ptr(cand_tok), _ptr(conf), _ptr(verdict),
            _ptr(selected), _ptr(num_commit), int(cand_seq.numel()), _ptr(accepted), wp, wb, _stream(stream)))

    def witness_workspace_bytes(self, B: int) -> int:
        return int(lib().epic_witness_workspace_bytes(self._h, int(B)))

    def witness(self, seqs, out_bytes, gap_len, status, witness_ws, workspace, stream=None):
        """epic_witness: out_bytes uint8 [B, bytes_per_seq], gap_len int32
        [B, max_gaps], status int32 [B]; witness_ws a uint8 tensor of
        witness_workspace_bytes(B) bytes."""
        B, n = int(seqs.shape[0]), int(seqs.shape[1])
        wp, wb = self._ws(workspace)
        wwp, wwb = self._ws(witness_ws)
        _check("epic_witness", lib().epic_witness(
            self._h, _ptr(seqs), B, n, _ptr(out_bytes), int(out_bytes.shape[1]), _ptr(gap_len), int(gap_len.shape[1]),
            _ptr(status), wwp, wwb, wp, wb, _stream(stream)))

    def work_counters(self, stream=None) -> np.ndarray:
        """int64[6]: walks, chart entries written, memo entries read, graph nodes,
        chart entries examined, chart entries used (read and cleared)."""
        out = np.zeros(6, dtype=np.int64)
        _check("epic_ctx_work_counters", lib().epic_ctx_work_counters(self._h, _stream(stream), out.ctypes.data))
        return out

    def set_timing(self, enable: bool = True):
        _check("epic_ctx_set_timing", lib().epic_ctx_set_timing(self._h, int(bool(enable))))

    def set_witness_lds(self, max_proofs: int = 8192, max_vis_words: int = 4096):
        _check("epic_ctx_set_witness_lds", lib().epic_ctx_set_witness_lds(self._h, int(max_proofs), int(max_vis_words)))

    def kernel_stats(self, stream=None) -> dict:
        """Per kernel kind (KERNEL_KINDS): summed event ms, launches and the
        int64[6] work counters of its walks (read and cleared)."""
        nk = len(KERNEL_KINDS)
        ms = np.zeros(nk, dtype=np.float64)
        n = np.zeros(nk, dtype=np.int64)
        work = np.zeros(6 * nk, dtype=np.int64)
        _check("epic_ctx_kernel_stats", lib().epic_ctx_kernel_stats(self._h, _stream(stream), ms.ctypes.data,
                                                                    n.ctypes.data, work.ctypes.data))
        return {k: {"ms": float(ms[i]), "launches": int(n[i]), "work": work[6 * i:6 * i + 6].copy()}
                for i, k in enumerate(KERNEL_KINDS)}

    @property
    def item_words(self) -> int:
        """32-bit words per item bitset of a chart entry."""
        return int(lib().epic_item_words(self._h))

    def device_error(self, stream=None) -> int:
        f = ctypes.c_uint32(0)
        _check("epic_ctx_device_error", lib().epic_ctx_device_error(self._h, _stream(stream), ctypes.byref(f)))
        return int(f.value)


def lds_stream(blocks: int, threads: int, iters: int, sink, stream=None):
    """Launch the LDS streaming microbenchmark (epic_diag_lds_stream) on a
    torch uint32 device tensor of 8 elements."""
    _check("epic_diag_lds_stream", lib().epic_diag_lds_stream(int(blocks), int(threads), int(iters), _ptr(sink),
                                                               _stream(stream)))


def clock_rates() -> tuple:
    """(shader clock kHz, wall clock kHz) of the current device."""
    a, b = ctypes.c_int32(0), ctypes.c_int32(0)
    _check("epic_diag_clock_rates", lib().epic_diag_clock_rates(ctypes.byref(a), ctypes.byref(b)))
    return int(a.value), int(b.value)
