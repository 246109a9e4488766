"""Move a drawn case onto a torch device (storage bits copied as they are)."""
import numpy as np
import torch


def to_torch(raw, dtype, device):
    """bf16 bit patterns (uint16) -> torch.bfloat16, binary32 -> torch.float32."""
    if raw is None:
        return None
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(raw).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(raw, dtype=np.float32))
    return t.to(device)


def from_torch(t):
    """Inverse of to_torch: bf16 -> uint16 bits, float32 -> float32 (numpy)."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def case_to_device(case, device="cuda"):
    """Dict of device tensors for a Case: X, Y, dY, A[], B[], idx, mask, segments."""
    dev = dict(
        X=to_torch(case.X, case.x_dtype, device),
        Y=to_torch(case.Y, case.y_dtype, device),
        dY=to_torch(case.dY, case.x_dtype, device),
        A=[to_torch(a, case.w_dtype, device) for a in case.A],
        B=[to_torch(b, case.w_dtype, device) for b in case.B],
        idx=torch.from_numpy(case.idx.astype(np.int32)).to(device),
        mask=None if case.mask is None else torch.from_numpy(case.mask.astype(np.uint8)).to(device),
    )
    if case.seg_offsets is not None:
        dev["seg_offsets"] = torch.from_numpy(case.seg_offsets.astype(np.int32)).to(device)
        dev["seg_adapter"] = torch.from_numpy(case.seg_adapter.astype(np.int32)).to(device)
    return dev
