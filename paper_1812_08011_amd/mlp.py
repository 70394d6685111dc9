"""One training step of a fully connected network in the paper's formats,
on the library's kernels (Sec. 2.1-2.2, Fig. 2; Sec. 3's recipe; the
speech DNN of the paper's experiments is 440 -> 1024 x 5 -> 6000).

Per step, for layers l = 0 .. L-1 with FP16 master weights W_l (fan_in x
fan_out), their FP8 copies and FP16 momentum buffers:

  forward, hidden layers: Z_l = chunk_gemm(A_l, W8_l) (FP16) and, in the same
    pass, Q8(Z_l); A_{l+1} = ReLU(Q8(Z_l)) in FP8 (relu_codes);
  last layer (Sec. 3: its GEMMs stay in FP16): A16 = ReLU(Z_{L-2}) in FP16,
    Y = chunk_gemm_p16(A16, W_{L-1});
  loss: squared error against the targets T; E = RN16((Y - T) * s) with
    s = loss_scale / batch (mse_grad_fp16) -- the loss scaling of Sec. 3;
  last layer backward in FP16: dA = chunk_gemm_p16(E, W^T),
    dW = chunk_gemm_p16(A16^T, E);
  hidden layers backward: E8_l = Q8(dA * [Z_l > 0]) (relu_backward_fp8),
    dW_l = chunk_gemm(A8_l^T, E8_l), dA = chunk_gemm(E8_l, W8_l^T);
  update: sr_weight_update of every layer (momentum, weight decay, stochastic
    rounding, FP8 copy for the hidden layers), with the loss scale removed
    through the scalars: lr / loss_scale and weight_decay * loss_scale (both
    FP32), so the momentum buffers hold loss-scaled values.

Random bits of the update of layer l at step t: Philox key = seed, offset =
t * L + l.  Everything is allocated once, in __init__ (device memory through
torch, the library's workspaces from its queries); step() only launches.
"""
import numpy as np

from . import (EXACT, chunk_gemm, chunk_gemm_fp8, chunk_gemm_fp8_workspace_size,
               chunk_gemm_p16, chunk_gemm_p16_workspace_size, chunk_gemm_workspace_size,
               fp8_quantize, lib, mse_grad_fp16, relu_backward_fp8, relu_codes,
               sr_weight_update)

SPEECH_DNN = (440, 1024, 1024, 1024, 1024, 1024, 6000)


class Fp8Mlp:
    def __init__(self, widths=SPEECH_DNN, batch=256, CL=64, mode=EXACT, device="cuda:0"):
        import torch
        lib()
        self.torch = torch
        self.widths = tuple(int(w) for w in widths)
        self.L = len(self.widths) - 1
        if self.L < 2:
            raise ValueError("need at least one hidden layer and the last layer")
        self.B, self.CL, self.mode, self.dev = int(batch), int(CL), int(mode), device
        u8 = lambda *s: torch.zeros(*s, dtype=torch.uint8, device=device)
        u16 = lambda *s: torch.zeros(*s, dtype=torch.uint16, device=device)
        B, L, w = self.B, self.L, self.widths
        self.W16 = [u16(w[l], w[l + 1]) for l in range(L)]
        self.V16 = [u16(w[l], w[l + 1]) for l in range(L)]
        self.W8 = [u8(w[l], w[l + 1]) for l in range(L - 1)]
        self.dW16 = [u16(w[l], w[l + 1]) for l in range(L)]
        self.A8 = [u8(B, w[l]) for l in range(L - 1)]          # A8[0] is the input
        self.Z16 = [u16(B, w[l + 1]) for l in range(L - 1)]
        self.Z8 = [u8(B, w[l + 1]) for l in range(L - 1)]
        self.A16 = u16(B, w[L - 1])
        self.Y16 = u16(B, w[L])
        self.E16 = u16(B, w[L])
        self.dA16 = [u16(B, w[l]) for l in range(L)]           # dA16[l]: error at A_l
        self.E8 = [u8(B, w[l + 1]) for l in range(L - 1)]
        # one workspace, large enough for every GEMM of the step
        need = [chunk_gemm_p16_workspace_size(0, 0, B, w[L], w[L - 1], CL),
                chunk_gemm_p16_workspace_size(0, 1, B, w[L - 1], w[L], CL),
                chunk_gemm_p16_workspace_size(1, 0, w[L - 1], w[L], B, CL)]
        for l in range(L - 1):
            need += [chunk_gemm_fp8_workspace_size(0, 0, B, w[l + 1], w[l], CL, mode),
                     chunk_gemm_workspace_size(1, 0, w[l], w[l + 1], B, CL, mode),
                     chunk_gemm_workspace_size(0, 1, B, w[l], w[l + 1], CL, mode)]
        self.ws_bytes = max(need)
        self.ws = u8(self.ws_bytes) if self.ws_bytes else None

    def macs(self):
        """Multiply-accumulates of one step (3 GEMMs per layer, no dA for the
        first layer)."""
        w, B = self.widths, self.B
        return sum((3 if l else 2) * B * w[l] * w[l + 1] for l in range(self.L))

    def set_weights(self, W16_codes):
        """FP16 master weights (numpy uint16 codes, one array per layer); the
        FP8 copies are their quantization, the momentum buffers start at 0."""
        torch = self.torch
        for l, Wc in enumerate(W16_codes):
            t = torch.from_numpy(np.ascontiguousarray(Wc, np.uint16).view(np.int16))
            self.W16[l].copy_(t.to(self.dev).view(torch.uint16))
            self.V16[l].zero_()
            if l < self.L - 1:
                fp8_quantize(self.W16[l], self.W8[l])

    def step(self, X8, T16, lr, momentum, weight_decay, loss_scale, seed, t):
        """X8: FP8 input (B x widths[0]); T16: FP16 targets (B x widths[-1])."""
        B, L, w, CL, mode, ws, wb = self.B, self.L, self.widths, self.CL, self.mode, self.ws, \
            self.ws_bytes
        self.A8[0].copy_(X8)
        for l in range(L - 1):
            chunk_gemm_fp8(0, 0, B, w[l + 1], w[l], CL, self.A8[l], w[l], self.W8[l], w[l + 1],
                           self.Z16[l], w[l + 1], self.Z8[l], w[l + 1], 1.0, mode, ws, wb)
            if l + 1 < L - 1:
                relu_codes(self.Z8[l], 8, self.A8[l + 1], B * w[l + 1])
        relu_codes(self.Z16[L - 2], 16, self.A16, B * w[L - 1])
        chunk_gemm_p16(0, 0, B, w[L], w[L - 1], CL, self.A16, w[L - 1], self.W16[L - 1], w[L],
                       self.Y16, w[L], ws, wb)
        s = float(np.float32(loss_scale) / np.float32(B))
        mse_grad_fp16(self.Y16, T16, self.E16, B * w[L], s)
        chunk_gemm_p16(0, 1, B, w[L - 1], w[L], CL, self.E16, w[L], self.W16[L - 1], w[L],
                       self.dA16[L - 1], w[L - 1], ws, wb)
        chunk_gemm_p16(1, 0, w[L - 1], w[L], B, CL, self.A16, w[L - 1], self.E16, w[L],
                       self.dW16[L - 1], w[L], ws, wb)
        for l in range(L - 2, -1, -1):
            relu_backward_fp8(self.dA16[l + 1], self.Z16[l], self.E8[l], B * w[l + 1], 1.0)
            chunk_gemm(1, 0, w[l], w[l + 1], B, CL, self.A8[l], w[l], self.E8[l], w[l + 1],
                       self.dW16[l], w[l + 1], mode, ws, wb)
            if l > 0:
                chunk_gemm(0, 1, B, w[l], w[l + 1], CL, self.E8[l], w[l + 1], self.W8[l],
                           w[l + 1], self.dA16[l], w[l], mode, ws, wb)
        lr_eff = float(np.float32(lr) / np.float32(loss_scale))
        wd_eff = float(np.float32(weight_decay) * np.float32(loss_scale))
        for l in range(L):
            sr_weight_update(self.W16[l], self.dW16[l], self.V16[l],
                             self.W8[l] if l < L - 1 else None, w[l] * w[l + 1], lr_eff,
                             momentum, wd_eff, seed, t * L + l)
        return self.Y16
