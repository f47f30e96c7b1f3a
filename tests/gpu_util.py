"""Helpers for the GPU tests: move a workload to the device and run the stage
through the C ABI."""
import numpy as np
import torch

from paper_2609_07536_amd import binding as B


def to_device(w, device="cuda"):
    x = torch.from_numpy(w.x_perm.view(np.int16)).to(device).view(torch.bfloat16)
    w2 = torch.from_numpy(w.w2.view(np.int16)).to(device).view(torch.bfloat16)
    off = torch.from_numpy(w.expert_offsets.astype(np.int32)).to(device)
    tid = torch.from_numpy(w.token_ids.astype(np.int32)).to(device)
    g = torch.from_numpy(w.gate_w.astype(np.float32)).to(device)
    return x, w2, off, tid, g


def run(w, C=-1, dev=None, workspace=None, counts=True, splits=None, trace=None,
        check_status=True, mode=None, out=None):
    """Returns (out numpy [T, H], C used, workspace).  mode None calls
    moe_gemm2_combine(_traced), else moe_gemm2_combine_ex with that mode."""
    dev = dev if dev is not None else to_device(w)
    x, w2, off, tid, g = dev
    cnt = w.counts if counts else None
    if workspace is None:
        wl, _ = B.make_workload(w.T, w.H, w.I, w.E, w.topk, splits or w.L,
                                rows=int(w.x_perm.shape[0]))
        workspace = B.Workspace(B.workspace_size(wl))
    out, c = B.combine(x, w2, off, tid, g, T=w.T, splits=splits or w.L, topk=w.topk,
                       counts=cnt, num_consumers=C, workspace=workspace, trace=trace,
                       mode=mode, out=out)
    torch.cuda.synchronize()
    if check_status:
        st = workspace.status()
        assert st == 0, f"device status {st}: {B.strerror(st)}"
    return out.cpu().numpy(), c, workspace
