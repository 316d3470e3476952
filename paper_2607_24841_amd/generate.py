"""Block-diffusion generation driver (Eq. (2)): prompt prefill, then per block
``steps`` calls of nmdlm_block_step that reveal ``k_unmask`` tokens each; a
finished block's keys/values stay in the caches as context.  The host only
loops and marshals; every step runs in libnmdlm's kernels and the token
state stays on the device until the end."""
from __future__ import annotations

import numpy as np
import torch

from . import binding as B


class Generator:
    def __init__(self, dm: B.DeviceModel, prompt_len: int, block: int):
        self.dm = dm
        self.B = block
        nb = max(B.nmdlm_block_step_workspace_size(dm, prompt_len, B.NMDLM_NO_HEAD),
                 B.nmdlm_block_step_workspace_size(dm, block, 0))
        self.ws = B.workspace(nb)
        self.tokens = torch.zeros(block, dtype=torch.int32, device="cuda")
        self.masked = torch.ones(block, dtype=torch.uint8, device="cuda")
        self.chosen = torch.zeros(block, dtype=torch.int32, device="cuda")

    def prefill(self, prompt_ids: torch.Tensor) -> int:
        P = int(prompt_ids.numel())
        masked = torch.zeros(P, dtype=torch.uint8, device="cuda")
        io = B.step_io(P, 0, pos0=0, flags=B.NMDLM_NO_HEAD, tokens=prompt_ids, masked=masked)
        B.nmdlm_block_step(self.dm, io, self.ws)
        return P

    def run_block(self, C: int, steps: int, k_unmask: int, log: list | None = None) -> torch.Tensor:
        self.tokens.zero_()
        self.masked.fill_(1)
        for _ in range(steps):
            io = B.step_io(self.B, C, pos0=C, flags=0, tokens=self.tokens, masked=self.masked,
                           k_unmask=k_unmask, unmasked_pos=self.chosen)
            B.nmdlm_block_step(self.dm, io, self.ws)
            if log is not None:
                log.append(self.chosen[:k_unmask].clone())
        return self.tokens.clone()

    def run(self, prompt_ids: torch.Tensor, n_blocks: int, steps: int, k_unmask: int,
            log: list | None = None) -> torch.Tensor:
        C = self.prefill(prompt_ids)
        out = []
        for _ in range(n_blocks):
            out.append(self.run_block(C, steps, k_unmask, log))
            C += self.B
        return torch.cat(out)


def generate(dm: B.DeviceModel, prompt: np.ndarray, n_blocks: int, block: int, steps: int,
             k_unmask: int):
    """Returns (generated ids [n_blocks*block], per-step chosen positions)."""
    g = Generator(dm, len(prompt), block)
    log: list = []
    ids = torch.from_numpy(np.asarray(prompt, dtype=np.int32)).cuda()
    out = g.run(ids, n_blocks, steps, k_unmask, log)
    torch.cuda.synchronize()
    return out.cpu().numpy(), [c.cpu().numpy() for c in log]
