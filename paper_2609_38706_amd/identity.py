"""Content identities of adapters and checkpoints (section 5.3: an adapter is bound by the identity
of its contents; section 6.5: the cost of computing it).  The tensors' bytes are packed into one
device pool (each tensor starting 4-byte aligned), their Merkle roots computed by the library's
kernels, and the identity formed from the tensors' metadata and roots by the library's host
routine; this module only arranges memory."""

from __future__ import annotations

from . import pkv_content_identity, pkv_tensor_roots, pkv_tree_work_bytes


class TensorPool:
    """Device pool of several tensors' bytes plus the buffers of one root pass."""

    def __init__(self, tensors, device="cuda"):
        import torch
        parts, starts, lens, pos = [], [], [], 0
        for t in tensors:
            b = t.detach().contiguous().reshape(-1).view(torch.uint8).to(device)
            starts.append(pos)
            lens.append(b.numel())
            parts.append(b)
            pad = (-b.numel()) % 256                                 # 256-byte aligned starts
            if pad:
                parts.append(torch.zeros(pad, dtype=torch.uint8, device=device))
            pos += b.numel() + pad
        self.data = torch.cat(parts) if parts else torch.zeros(0, dtype=torch.uint8, device=device)
        self.n = len(tensors)
        self.nbytes = lens
        self.off = torch.tensor(starts or [0], dtype=torch.int64, device=device)
        self.len = torch.tensor(lens or [0], dtype=torch.int64, device=device)
        work = pkv_tree_work_bytes(self.data.numel(), self.n)
        self.work = torch.empty(max(1, (work + 7) // 8), dtype=torch.int64, device=device)
        self.roots = torch.empty((max(1, self.n), 32), dtype=torch.uint8, device=device)
        self.status = torch.zeros(1, dtype=torch.int32, device=device)

    def compute_roots(self, stream=None):
        """Enqueues the root pass (asynchronous)."""
        pkv_tensor_roots(self.data, self.off[: self.n], self.len[: self.n], self.work, self.roots, self.status, stream)

    def host_roots(self):
        if int(self.status.item()) != 0:
            raise RuntimeError(f"tensor roots failed on the device: status {int(self.status.item())}")
        return [bytes(r) for r in self.roots[: self.n].cpu().numpy()]


def content_identity(named_tensors, config=(), device="cuda") -> bytes:
    """named_tensors: (name bytes, torch tensor) pairs; the dtype recorded is the tensor's torch dtype
    name, the shape its shape.  Returns the 32-byte identity."""
    pool = TensorPool([t for _, t in named_tensors], device)
    pool.compute_roots()
    roots = pool.host_roots()
    recs = [(bytes(n), str(t.dtype).replace("torch.", "").encode(), tuple(t.shape), nb, r)
            for (n, t), nb, r in zip(named_tensors, pool.nbytes, roots)]
    return pkv_content_identity(recs, config)
