"""Convenience object around the C ABI: owns the device coefficient buffer of
one model (all type pairs) and allocates outputs as torch tensors.  All
arithmetic happens in libdpc (host table builder, HIP kernels)."""
import numpy as np
import torch

from . import binding as B

_TORCH = {B.DPC_F64: (torch.float64, torch.float64),
          B.DPC_F32: (torch.float32, torch.float32),
          B.DPC_F32_ACC64: (torch.float32, torch.float64)}   # (storage, accumulate/output)


class SeATab:
    """Compressed se_a descriptor of one model.

    nets     per ordered type pair alpha*ntypes+beta: {"W": [...], "b": [...]}
    lo, L1, L2  per pair table ranges; d1, d2 strides (scalars)
    sel      neighbours per type; m2 = M' rows used by D."""

    def __init__(self, nets, lo, L1, L2, d1, d2, sel, m2, dtype=B.DPC_F64, device="cuda"):
        self.ntypes = len(sel)
        npair = self.ntypes ** 2
        if len(nets) != npair:
            raise ValueError("need one net per ordered type pair")
        self.sel = [int(s) for s in sel]
        self.nnei = sum(self.sel)
        self.m1 = int(np.asarray(nets[0]["W"][-1]).shape[1])
        self.m2 = int(m2)
        self.dtype = dtype
        self.t_in, self.t_acc = _TORCH[dtype]
        self.ranges = B.make_ranges(lo, [d1] * npair, L1, [d2] * npair, L2)
        self.host_coeff = B.build_tables(nets, self.ranges, dtype)
        self.coeff = torch.from_numpy(self.host_coeff).to(device)
        self.device = device

    def forward(self, em, nlist, atype, T=None, D=None, stream=None):
        nloc = nlist.shape[0]
        if T is None:
            T = torch.empty((nloc, self.m1, 4), dtype=self.t_acc, device=self.device)
        if D is None:
            D = torch.empty((nloc, self.m1, self.m2), dtype=self.t_acc, device=self.device)
        self._check(em, nlist, atype)
        B.dpc_se_a_tab_fwd(stream or torch.cuda.current_stream(), self.dtype, nloc, self.ntypes,
                           self.sel, self.m1, self.m2, self.ranges, self.coeff, atype, nlist, em,
                           T, D)
        return T, D

    def backward(self, em, nlist, atype, dT, dR=None, stream=None):
        nloc = nlist.shape[0]
        if dR is None:
            dR = torch.empty((nloc, self.nnei, 4), dtype=self.t_acc, device=self.device)
        self._check(em, nlist, atype)
        if dT.dtype != self.t_in or tuple(dT.shape) != (nloc, self.m1, 4):
            raise ValueError("dE/dT has the wrong dtype or shape")
        B.dpc_se_a_tab_bwd(stream or torch.cuda.current_stream(), self.dtype, nloc, self.ntypes,
                           self.sel, self.m1, self.ranges, self.coeff, atype, nlist, em, dT, dR)
        return dR

    def backward_from_dD(self, em, nlist, atype, T, dD, dR=None, stream=None):
        """dE/dR~ from dE/dD and the forward's T in one call (the descriptor
        backward fused into the backward; float64, M1 <= 128, even M' <= 16)."""
        nloc = nlist.shape[0]
        if dR is None:
            dR = torch.empty((nloc, self.nnei, 4), dtype=self.t_acc, device=self.device)
        self._check(em, nlist, atype)
        if T.dtype != torch.float64 or tuple(T.shape) != (nloc, self.m1, 4):
            raise ValueError("T has the wrong dtype or shape")
        if dD.dtype != torch.float64 or tuple(dD.shape) != (nloc, self.m1, self.m2):
            raise ValueError("dE/dD has the wrong dtype or shape")
        B.dpc_se_a_tab_bwd_from_dD(stream or torch.cuda.current_stream(), self.dtype, nloc, self.ntypes,
                                   self.sel, self.m1, self.m2, self.ranges, self.coeff, atype, nlist, em,
                                   T, dD, dR)
        return dR

    def descriptor_backward(self, T, dD, dT=None, stream=None):
        """dE/dT from dE/dD and the forward's T (the input dtype of backward())."""
        nloc = T.shape[0]
        if T.dtype != self.t_acc or tuple(T.shape) != (nloc, self.m1, 4):
            raise ValueError("T has the wrong dtype or shape")
        if dD.dtype != self.t_acc or tuple(dD.shape) != (nloc, self.m1, self.m2):
            raise ValueError("dE/dD has the wrong dtype or shape")
        if dT is None:
            dT = torch.empty((nloc, self.m1, 4), dtype=self.t_in, device=self.device)
        B.dpc_descriptor_bwd(stream or torch.cuda.current_stream(), self.dtype, nloc, self.m1,
                             self.m2, T, dD, dT)
        return dT

    def _check(self, em, nlist, atype):
        nloc = nlist.shape[0]
        if em.dtype != self.t_in or tuple(em.shape) != (nloc, self.nnei, 4):
            raise ValueError("R~ has the wrong dtype or shape")
        if nlist.dtype != torch.int32 or tuple(nlist.shape) != (nloc, self.nnei):
            raise ValueError("nlist must be int32 [nloc, nnei]")
        if atype.dtype != torch.int32 or tuple(atype.shape) != (nloc,):
            raise ValueError("atype must be int32 [nloc]")
