"""Encoder-decoder block diffusion driver (Sec. III-A, Eqs. (5)-(6)) over the
C ABI: the first n_enc layers of a model are the encoder, the others the
decoder.  The encoder runs block-causally: the prompt once, then every
finished block over the cached context plus itself (each token passes the
encoder once).  After each encoder pass every decoder layer, as a one-layer
model, runs over the encoder output to write the keys and values of those
positions into its caches.  A block is ``steps`` decoder block steps with
the head, revealing ``k_unmask`` tokens each.  The host only loops and
marshals; every step runs in libnmdlm's kernels and the tokens stay on the
device."""
from __future__ import annotations

import torch

from . import binding as B


class E2D2:
    def __init__(self, dm: B.DeviceModel, n_enc: int, prompt_len: int, n_blocks: int, block: int):
        n_dec = len(dm.layers) - n_enc
        if n_enc < 0 or n_dec < 1:
            raise ValueError("need 0 <= n_enc < number of layers")
        total = prompt_len + n_blocks * block
        if dm.cache_cap < total:
            raise ValueError("cache capacity below the prompt plus the blocks")
        self.dm, self.n_enc, self.B = dm, n_enc, block
        self.enc = dm.view(0, n_enc, head=False)
        self.dec = dm.view(n_enc, n_dec, head=True)
        self.dec_layers = [dm.view(n_enc + l, 1, head=False) for l in range(n_dec)]
        mx = max(prompt_len, block)
        nb = max(B.nmdlm_block_step_workspace_size(self.enc, mx, B.NMDLM_NO_HEAD),
                 B.nmdlm_block_step_workspace_size(self.dec_layers[0], mx, B.NMDLM_NO_HEAD),
                 B.nmdlm_block_step_workspace_size(self.dec, block, 0))
        self.ws = B.workspace(nb)
        self.h = torch.empty(dm.T * mx * (dm.d // 64), dtype=torch.int64, device="cuda")
        self.ctx = torch.zeros(total, dtype=torch.int32, device="cuda")
        self.ctx_masked = torch.zeros(total, dtype=torch.uint8, device="cuda")
        self.tokens = torch.zeros(block, dtype=torch.int32, device="cuda")
        self.masked = torch.ones(block, dtype=torch.uint8, device="cuda")
        self.chosen = torch.zeros(block, dtype=torch.int32, device="cuda")

    def _h(self, M: int) -> torch.Tensor:
        return self.h[:self.dm.T * M * (self.dm.d // 64)].view(self.dm.T, M, self.dm.d // 64)

    def encode(self, C: int, M: int) -> None:
        """Encoder over context tokens [C, C+M) (attending to the cached
        [0, C) and to themselves), then every decoder layer's keys and values
        of those positions from the encoder output."""
        io = B.step_io(M, C, pos0=C, flags=B.NMDLM_NO_HEAD, tokens=self.ctx[C:C + M],
                       masked=self.ctx_masked[C:C + M], y_out=self._h(M))
        B.nmdlm_block_step(self.enc, io, self.ws)
        for v in self.dec_layers:
            B.nmdlm_block_step(v, B.step_io(M, C, pos0=C, flags=B.NMDLM_NO_HEAD, x_in=self._h(M)),
                               self.ws)

    def denoise(self, C: int, steps: int, k_unmask: int, log: list | None = None) -> None:
        """z_{s+1} = f_dec(z_s, h^b) for ``steps`` steps (Eq. (6)) on the block at
        [C, C+B); its tokens then join the context."""
        self.tokens.zero_()
        self.masked.fill_(1)
        for _ in range(steps):
            io = B.step_io(self.B, C, pos0=C, flags=0, tokens=self.tokens, masked=self.masked,
                           k_unmask=k_unmask, unmasked_pos=self.chosen)
            B.nmdlm_block_step(self.dec, io, self.ws)
            if log is not None:
                log.append(self.chosen[:k_unmask].clone())
        self.ctx[C:C + self.B].copy_(self.tokens)

    def generate(self, P: int, n_blocks: int, steps: int, k_unmask: int,
                 log: list | None = None) -> int:
        """Prompt already in ctx[:P]; returns the final context length."""
        self.encode(0, P)
        C = P
        for _ in range(n_blocks):
            self.denoise(C, steps, k_unmask, log)
            self.encode(C, self.B)
            C += self.B
        return C


def e2d2_generate(dm: B.DeviceModel, n_enc: int, prompt, n_blocks: int, block: int, steps: int,
                  k_unmask: int):
    """Returns (generated ids [n_blocks*block], per-step chosen positions)."""
    import numpy as np
    P = len(prompt)
    g = E2D2(dm, n_enc, P, n_blocks, block)
    g.ctx[:P].copy_(torch.from_numpy(np.asarray(prompt, dtype=np.int32)))
    log: list = []
    C = g.generate(P, n_blocks, steps, k_unmask, log)
    torch.cuda.synchronize()
    return g.ctx[P:C].cpu().numpy(), [c.cpu().numpy() for c in log]
