"""Block-diffusion generation driver (Eq. (2)): prompt prefill, then per block
``steps`` calls of nmdlm_block_step that reveal ``k_unmask`` tokens each; a
finished block's keys/values stay in the caches as context.  The host only
loops and marshals; every step runs in libnmdlm's kernels and the token
state stays on the device until the end.  Several sequences (prompts of
one length) advance together, one batched step per denoising step."""
from __future__ import annotations

import numpy as np
import torch

from . import binding as B


class Generator:
    def __init__(self, dm: B.DeviceModel, prompt_len: int, block: int, n_seq: int = 1):
        self.dm = dm
        self.B = block
        self.n = n_seq
        nb = max(B.nmdlm_block_step_workspace_size(dm, n_seq * prompt_len, B.NMDLM_NO_HEAD),
                 B.nmdlm_block_step_workspace_size(dm, n_seq * block, 0))
        self.ws = B.workspace(nb)
        self.tokens = torch.zeros(n_seq * block, dtype=torch.int32, device="cuda")
        self.masked = torch.ones(n_seq * block, dtype=torch.uint8, device="cuda")
        self.chosen = torch.zeros((n_seq, block), dtype=torch.int32, device="cuda")

    def prefill(self, prompt_ids: torch.Tensor) -> int:
        """prompt_ids: the n_seq prompts one after the other."""
        P = int(prompt_ids.numel()) // self.n
        masked = torch.zeros(self.n * P, dtype=torch.uint8, device="cuda")
        io = B.step_io(P, 0, pos0=0, flags=B.NMDLM_NO_HEAD, tokens=prompt_ids, masked=masked,
                       n_seq=self.n)
        B.nmdlm_block_step(self.dm, io, self.ws)
        return P

    def run_block(self, C: int, steps: int, k_unmask: int, log: list | None = None) -> torch.Tensor:
        self.tokens.zero_()
        self.masked.fill_(1)
        # chosen positions: [n_seq][k_unmask] packed at the front of the buffer
        chosen_k = self.chosen.view(-1)[:self.n * k_unmask].view(self.n, k_unmask)
        for _ in range(steps):
            io = B.step_io(self.B, C, pos0=C, flags=0, tokens=self.tokens, masked=self.masked,
                           k_unmask=k_unmask, unmasked_pos=self.chosen, n_seq=self.n)
            B.nmdlm_block_step(self.dm, io, self.ws)
            if log is not None:
                log.append(chosen_k.clone())
        return self.tokens.view(self.n, self.B).clone()

    def run(self, prompt_ids: torch.Tensor, n_blocks: int, steps: int, k_unmask: int,
            log: list | None = None) -> torch.Tensor:
        """Generated ids [n_seq][n_blocks * block]."""
        C = self.prefill(prompt_ids)
        out = []
        for _ in range(n_blocks):
            out.append(self.run_block(C, steps, k_unmask, log))
            C += self.B
        return torch.cat(out, dim=1)


def generate(dm: B.DeviceModel, prompt: np.ndarray, n_blocks: int, block: int, steps: int,
             k_unmask: int):
    """Returns (generated ids [n_blocks*block], per-step chosen positions)."""
    ids, log = generate_batch(dm, np.asarray(prompt)[None, :], n_blocks, block, steps, k_unmask)
    return ids[0], [c[0] for c in log]


def generate_batch(dm: B.DeviceModel, prompts: np.ndarray, n_blocks: int, block: int, steps: int,
                   k_unmask: int):
    """prompts [n_seq][P] advanced together (one batched step per denoising
    step).  Returns (generated ids [n_seq][n_blocks*block], per-step chosen
    positions [n_seq][k_unmask])."""
    prompts = np.asarray(prompts, dtype=np.int32)
    n, P = prompts.shape
    g = Generator(dm, P, block, n_seq=n)
    log: list = []
    ids = torch.from_numpy(np.ascontiguousarray(prompts).reshape(-1)).cuda()
    out = g.run(ids, n_blocks, steps, k_unmask, log)
    torch.cuda.synchronize()
    return out.cpu().numpy(), [c.cpu().numpy() for c in log]
