"""GPU-side helpers for parity tests: run the C-ABI library on numpy inputs."""
from __future__ import annotations

import numpy as np

from paper_2606_00722_amd import epic
from paper_2606_00722_amd import workloads as W


class Gpu:
    def __init__(self, arrays: W.Arrays, max_batch: int, max_seq: int, max_cands: int):
        import torch

        self.torch = torch
        self.dev = torch.device("cuda:0")
        self.ctx = epic.Context.from_problem(arrays, max_batch, max_seq, max_cands)
        self.ctx.lexmemo_build()
        self.ws = self.ctx.alloc_workspace(self.dev)
        self.counts = torch.zeros(2, dtype=torch.int64, device=self.dev)

    def t(self, a, dt=None):
        torch = self.torch
        return torch.from_numpy(np.ascontiguousarray(a)).to(self.dev, dt or torch.int32)

    def validate(self, seqs, seq, pos, tok) -> np.ndarray:
        torch = self.torch
        C = len(seq)
        out = torch.full((max(C, 1),), 7, dtype=torch.uint8, device=self.dev)
        self.ctx.validate(self.t(seqs), self.t(seq), self.t(pos), self.t(tok), out[:C], self.ws)
        torch.cuda.synchronize()
        return out[:C].cpu().numpy()

    def select(self, seqs, seq, pos, tok, conf, verdict):
        torch = self.torch
        C = len(seq)
        out = torch.full((max(C, 1),), 7, dtype=torch.uint8, device=self.dev)
        self.counts.zero_()
        self.ctx.select(self.t(seqs), self.t(seq), self.t(pos), self.t(tok), self.t(conf, torch.float32),
                        self.t(verdict, torch.uint8), out[:C], self.ws, counts=self.counts)
        torch.cuda.synchronize()
        return out[:C].cpu().numpy(), tuple(int(x) for x in self.counts.cpu().tolist())

    def errors(self) -> int:
        return self.ctx.device_error()

    def fallback(self, seqs, seq, pos, tok, conf, verdict, selected, num_commit) -> np.ndarray:
        torch = self.torch
        C = len(seq)
        out = torch.full((max(C, 1),), 7, dtype=torch.uint8, device=self.dev)
        self.ctx.fallback(self.t(seqs), self.t(seq), self.t(pos), self.t(tok), self.t(conf, torch.float32),
                          self.t(verdict, torch.uint8), self.t(selected, torch.uint8), self.t(num_commit),
                          out[:C], self.ws)
        torch.cuda.synchronize()
        return out[:C].cpu().numpy()
