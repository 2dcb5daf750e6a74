"""The DeiT encoder with the pruned linear layers in place, chained on the GPU.

Composition only: every step is one liblpv call (lpv.py), nothing is computed
here.  The paper prunes the four linear layers of every DeiT encoder block
(qkv, proj, fc1, fc2; Sec. 4) and compares whole-model inference (Tab. 2);
this chains the standard pre-norm block around them:

    A = LN(x)
    per block:  qkv = A Wqkv~^T + b         (block-sparse or dense)
                O   = attention(qkv)         (H heads of 64)
                P   = O Wproj~^T + b
                x   = x + P;  A = LN(x)
                Hd  = GELU(A Wfc1~^T + b)
                P   = Hd Wfc2~^T + b
                x   = x + P;  A = LN(x)      (the next block's first LN)

Every layer norm uses the same gamma / beta.  The residual stream alternates
between two buffers, so a run never overwrites its own input and every run
computes the same function of ``x0``.
"""
import torch

from . import lpv


class Linear:
    """One linear layer of the chain on the device: the dense weight, its
    packed block-sparse handle (None until packed), bias and epilogue."""

    def __init__(self, name, W, mask, bias, b_r, b_c, gelu):
        self.name, self.W, self.mask, self.bias = name, W, mask, bias
        self.b_r, self.b_c, self.gelu = b_r, b_c, gelu
        self.h = lpv.bsr_pack(W, mask, b_r, b_c)

    def __call__(self, x, y, sparse):
        epi = "gelu" if self.gelu else None
        if sparse:
            return lpv.bsr_linear(self.h, x, self.bias, y, epi=epi)
        return lpv.dense_linear(self.W, x, self.bias, y, epi=epi)

    def close(self):
        self.h.close()


class EncoderChain:
    """``blocks`` DeiT encoder blocks over M = n_seq * T tokens of width D.

    linears: 4 * blocks Linear objects in the order (qkv, proj, fc1, fc2) per
    block; gamma, beta: the layer norms' D-element parameters."""

    def __init__(self, linears, n_seq, T, H, gamma, beta, eps=1e-6):
        if len(linears) % 4:
            raise ValueError("four linear layers per block")
        self.linears, self.n_seq, self.T, self.H = linears, n_seq, T, H
        self.gamma, self.beta, self.eps = gamma, beta, eps
        D = linears[0].W.shape[1]
        M = n_seq * T
        dt, dv = gamma.dtype, gamma.device
        new = lambda cols: torch.empty((M, cols), dtype=dt, device=dv)
        self.D, self.M = D, M
        self.A, self.O, self.P = new(D), new(D), new(D)
        self.qkv, self.Hd = new(linears[0].W.shape[0]), new(linears[2].W.shape[0])
        self.R = [new(D), new(D)]

    @property
    def blocks(self):
        return len(self.linears) // 4

    def run(self, x0, sparse=True, trace=None, linear_events=None):
        """One forward pass from the token activations x0 (M x D).  Returns
        (x, A): the residual stream after the last block and its layer norm.

        trace(name, inputs, output), if given, is called after every step with
        the step's input tensors (a dict) and its output, for checking a link
        at a time.  linear_events, if a list, receives a (start, end) pair of
        timing events recorded around every linear launch."""
        g, b, eps = self.gamma, self.beta, self.eps
        A, O, P, qkv, Hd, R = self.A, self.O, self.P, self.qkv, self.Hd, self.R

        def lin(layer, x, y):
            if linear_events is not None:
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                layer(x, y, sparse)
                e1.record()
                linear_events.append((e0, e1))
            else:
                layer(x, y, sparse)
            if trace:
                trace(layer.name, {"x": x}, y)

        x, nxt = x0, 0
        lpv.add_layernorm(x, None, g, b, eps, out=A)
        if trace:
            trace("ln.in", {"x": x}, A)
        for blk in range(self.blocks):
            q, pr, f1, f2 = self.linears[4 * blk:4 * blk + 4]
            lin(q, A, qkv)
            lpv.attention(qkv, self.n_seq, self.T, self.H, out=O)
            if trace:
                trace("%d.attention" % blk, {"qkv": qkv}, O)
            lin(pr, O, P)
            lpv.add_layernorm(x, P, g, b, eps, S=R[nxt], out=A)
            if trace:
                trace("%d.add_ln1" % blk, {"x": x, "y": P, "s": R[nxt]}, A)
            x, nxt = R[nxt], 1 - nxt
            lin(f1, A, Hd)
            lin(f2, Hd, P)
            lpv.add_layernorm(x, P, g, b, eps, S=R[nxt], out=A)
            if trace:
                trace("%d.add_ln2" % blk, {"x": x, "y": P, "s": R[nxt]}, A)
            x, nxt = R[nxt], 1 - nxt
        return x, A

    def capture(self, x0, sparse=True):
        """The forward pass from x0 captured once into a HIP graph (through
        torch.cuda.CUDAGraph): replaying it relaunches the same 1 + 6 * blocks
        kernels on the same buffers with no host work per launch.  Every call
        of the chain is capturable (no allocation, no host synchronisation, no
        memset); one eager pass first settles the kernels' one-time set-up.
        Returns (graph, (x, A)): the outputs the replays rewrite."""
        self.run(x0, sparse)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            out = self.run(x0, sparse)
        torch.cuda.synchronize()
        return graph, out

    def close(self):
        for layer in self.linears:
            layer.close()


def deit_chain(layers, to_dev, n_seq, T=197, H=12, eps=1e-6):
    """An EncoderChain from generated layer inputs (objects with W, mask, bias,
    b_r, b_c, gelu, name as numpy arrays; ``to_dev`` moves an array of the
    element type to the GPU).  Layer norms: gamma = 1, beta = 0."""
    lins = [Linear(w.name, to_dev(w.W), torch.from_numpy(w.mask).cuda(), to_dev(w.bias),
                   w.b_r, w.b_c, w.gelu) for w in layers]
    D = lins[0].W.shape[1]
    dt = lins[0].W.dtype
    gamma = torch.ones(D, dtype=dt, device="cuda")
    beta = torch.zeros(D, dtype=dt, device="cuda")
    return EncoderChain(lins, n_seq, T, H, gamma, beta, eps)
