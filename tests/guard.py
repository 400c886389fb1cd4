"""Guard bands for device buffers written by the HIP path.

A buffer is allocated with GUARD extra elements before and after the part
handed to the library; both bands hold a NaN with a fixed payload.  After
the call the bands must be bit-identical: a kernel that writes past either
end of its output changes them."""
import numpy as np

GUARD = 64                   # elements per band (256 bytes: keeps 16-byte alignment)
PATTERN = np.int32(0x7FC0DEAD)  # a quiet NaN with a payload


def guarded(shape, dtype=None, fill=None, device="cuda"):
    """(view, full): view has `shape`, full = band | view | band."""
    import torch
    dtype = dtype or torch.float32
    assert dtype in (torch.float32, torch.int32)
    n = int(np.prod(shape))
    full = torch.empty(n + 2 * GUARD, dtype=torch.int32, device=device)
    full.fill_(int(PATTERN))
    view = full[GUARD:GUARD + n].view(dtype).view(*shape)
    if fill is not None:
        view.copy_(fill)
    return view, full


def check_guards(full, name="buffer"):
    import torch
    band = torch.cat([full[:GUARD], full[-GUARD:]]).cpu().numpy()
    bad = np.nonzero(band != PATTERN)[0]
    assert bad.size == 0, f"{name}: guard band overwritten at {bad[:8].tolist()}"
