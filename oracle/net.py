"""Multi-stage PETRA schedule on a RevNet-shaped network (Alg. 1, Eq. 5,
Sec. 3.2 "Non-reversible stages", App. B delays).

Network (CIFAR-style RevNet, Sec. 4.1 "Model adaptations"): a 3x3 stem
(conv-BN-ReLU, no max-pool), then J stages of reversible blocks whose width
doubles from stage to stage; between stages a non-reversible downsampling
(conv1x1 stride 2 + BN) opens the next stage; the last stage ends with global
average pooling, a linear layer with bias and softmax cross-entropy averaged
over the micro-batch.  Readings: stage 0 = stem + blocks, stage j > 0 =
downsampling + blocks, the last stage also owns the head; the stem has a ReLU
after its BN, the downsampling has none; the downsampling convolves the two
streams as one tensor (x1 first) and its output is split into halves again.

The linear head reads the fp32 master weights (it is not a convolution and
has no lower-precision compute copy); `weight_view` applies to conv weights.
`store` (identity by default) holds activations and activation gradients at a
storage precision where the method materialises them, as in revblock: the
front conv output, its BN(+ReLU) output, the block tensors, and the front
layer's gradients.

Schedule (0-based stage index j, J stages, one hop per tick): at tick t stage j
runs the forward of micro-batch t - j and the backward of micro-batch
t - (2J - 2 - j), so the delay between a stage's forward and backward of the
same micro-batch is 2(J - 1 - j), i.e. 2(J - j) with the paper's 1-based j.
Every forward and backward of a tick reads the stage's current parameters and
the update follows both (Eq. 5).  The last stage computes the loss and its own
backward in the same tick.  Non-reversible front layers keep their input in a
buffer and recompute it on the backward, discarding the reconstructed input
that arrives from above; stage 0 re-reads its images from the dataset
(Alg. 1; Sec. 4.2).  A reversible stage sends back its reconstructed input; a
stage with a buffer sends back the buffered input (Alg. 1, reading of the
backward send).

Buffer variants (Table 4 and App. B): every stage may also keep, per
micro-batch in flight, the parameters its forward used (parameter buffer,
PipeDream-style weight stash) and its blocks' input (input buffer).  The
backward then uses, with `use_inputs`, the stored block input instead of the
reconstruction and, with `use_params`, the stashed parameters for the
Jacobians (blocks and front layer).  With a parameter buffer but no input
buffer the input is reconstructed with the latest parameters and the VJP taken
at the reconstruction with the stashed ones (reading of the fourth line of
Table 4: reconstruction with the latest parameters, the delayed ones for the
Jacobian; "the input" is the stage's block input).  Both switches on give the
standard delayed gradient of the method's analysis (App. B); both off is PETRA.
The last stage runs its forward and backward in the same tick, so all four
variants coincide there.
"""
from __future__ import annotations

import copy
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

from . import bn, conv, revblock, sgd


def _identity(a):
    return a


def nonrev_forward(x, w, g, b, eps, stride, relu, store=_identity):
    h = store(conv.forward(x, w, stride=stride, pad=(w.shape[1] - 1) // 2))
    o, cache = bn.forward(h, g, b, eps)
    a = store(np.maximum(o, 0.0) if relu else o)
    return a, (x, h, o, cache)


def nonrev_vjp(d, w, g, graph, stride, relu, store=_identity):
    x, _, o, cache = graph
    if relu:
        d = d * (o > 0.0)
    dh, dg, db = bn.backward(d, cache, g)
    dh = store(dh)
    pad = (w.shape[1] - 1) // 2
    return store(conv.dgrad(dh, w, x.shape, stride=stride, pad=pad)), (
        conv.wgrad(x, dh, w.shape, stride=stride, pad=pad), dg, db)


def head_loss(x, wfc, bfc, labels):
    """Global average pool -> linear -> softmax cross-entropy (batch mean)."""
    pooled = x.mean(axis=(1, 2))                      # [N, C]
    logits = pooled @ wfc.T + bfc                     # [N, K]
    z = logits - logits.max(axis=1, keepdims=True)
    lse = np.log(np.exp(z).sum(axis=1))
    n = x.shape[0]
    loss = float(np.mean(lse - z[np.arange(n), labels]))
    return loss, (x.shape, pooled, z, lse)


def head_vjp(wfc, labels, cache):
    shape, pooled, z, lse = cache
    n = shape[0]
    p = np.exp(z - lse[:, None])
    p[np.arange(n), labels] -= 1.0
    dlogits = p / n
    dw = dlogits.T @ pooled
    db = dlogits.sum(axis=0)
    dpooled = dlogits @ wfc
    dx = np.broadcast_to(dpooled[:, None, None, :] / (shape[1] * shape[2]), shape).copy()
    return dx, dw, db


class NetStage:
    """One stage: an optional non-reversible front layer (`front` = "stem" on the
    images or "trans" for a downsampling, None for a purely reversible stage),
    `blocks` reversible blocks (possibly none) and, for the last stage, the head.
    Parameter order: front (w, gamma, beta), blocks, head (weight, bias)."""

    def __init__(self, params, names, first: bool, last: bool, blocks: int, eps: float,
                 bn_momentum: float, dtype, weight_view, store=None, front="auto"):
        self.params = [np.array(p, dtype=dtype) for p in params]
        self.names = list(names)
        self.front = ("stem" if first else "trans") if front == "auto" else front
        self.first, self.last, self.blocks = first, last, blocks
        self.fo = 3 if self.front else 0     # first block parameter
        self.ro = 1 if self.front else 0     # first block BN slot
        self.eps, self.bn_momentum, self.dtype = eps, bn_momentum, dtype
        self.weight_view = weight_view
        if store is None:
            self.store = _identity
        else:
            self.store = lambda a: np.asarray(store(np.asarray(a, np.float32)), dtype=dtype)
        self.accum = [np.zeros_like(p) for p in self.params]
        self.buf = [np.zeros_like(p) for p in self.params]
        nbn = self.ro + blocks * 4
        self.run_mean = [np.zeros(self.params[3 * i + 1].shape, dtype) for i in range(nbn)]
        self.run_var = [np.ones(self.params[3 * i + 1].shape, dtype) for i in range(nbn)]
        self.t = 0
        self.buffer: Dict[int, tuple] = {}
        self.stash: Dict[int, list] = {}     # parameter buffer: micro-batch -> parameters
        self.inbuf: Dict[int, tuple] = {}    # input buffer: micro-batch -> block input

    def _w(self, i, P=None):
        w = (self.params if P is None else P)[i]
        if self.weight_view is not None:
            w = np.asarray(self.weight_view(w.astype(np.float32)), dtype=self.dtype)
        return w

    def _layers(self, b, f, P=None):
        P = self.params if P is None else P
        base = self.fo + (2 * b + f) * 6
        return [(self._w(base + 3 * l, P), P[base + 3 * l + 1], P[base + 3 * l + 2])
                for l in range(2)]

    def _front(self, x1, x2, P=None):
        P = self.params if P is None else P
        stem = self.front == "stem"
        x = x1 if stem else np.concatenate([x1, x2], axis=-1)
        stride = 1 if stem else 2
        a, graph = nonrev_forward(x, self._w(0, P), P[1], P[2], self.eps,
                                  stride, relu=stem, store=self.store)
        c = a.shape[-1] // 2
        return a[..., :c], a[..., c:], graph

    def forward(self, x1, x2, m=None):
        if m is not None:
            self.stash[m] = [p.copy() for p in self.params]
        y1, y2 = self._front(x1, x2)[:2] if self.front else (x1, x2)
        if m is not None:
            self.inbuf[m] = (y1, y2)
        for b in range(self.blocks):
            y1, y2 = revblock.block_forward(y1, y2, self._layers(b, 0), self._layers(b, 1), self.eps,
                                            self.store)
        return y1, y2

    def _running(self, slot, stats):
        cache, m = stats
        self.run_mean[slot], self.run_var[slot] = bn.running_update(
            self.run_mean[slot], self.run_var[slot], cache, m, self.bn_momentum)

    def backward(self, y1, y2, g1, g2, x1, x2, k, m=None, use_inputs=False, use_params=False):
        """Blocks: reconstruct + VJP from (y, g) (PETRA), or one of the buffer
        variants for micro-batch m (see the module notes).  Front: recompute
        from the buffered input (x1, x2) and VJP.  Returns the input gradient
        halves and the parameter gradients."""
        stash = self.stash.pop(m, None) if m is not None else None
        inbuf = self.inbuf.pop(m, None) if m is not None else None
        P = stash if use_params else self.params
        grads: List[Optional[np.ndarray]] = [None] * len(self.params)

        def take(b, r):
            for f, key in ((0, "dF"), (1, "dG")):
                base = self.fo + (2 * b + f) * 6
                stats = r["stats_F" if f == 0 else "stats_G"]
                for l, (dw, dg, db) in enumerate(r[key]):
                    grads[base + 3 * l: base + 3 * l + 3] = [dw, dg, db]
                    self._running(self.ro + (base - self.fo + 3 * l) // 3, stats[l])

        if not use_inputs and not use_params:
            for b in reversed(range(self.blocks)):
                r = revblock.block_reconstruct_vjp(y1, y2, g1, g2, self._layers(b, 0),
                                                   self._layers(b, 1), self.eps, self.store)
                take(b, r)
                y1, y2, g1, g2 = r["x1"], r["x2"], r["dx1"], r["dx2"]
            self.last_used = dict(u=(y1, y2), P=list(P))
        else:
            if use_inputs:
                u1, u2 = inbuf
            else:   # reconstruction with the latest parameters
                u1, u2 = y1, y2
                for b in reversed(range(self.blocks)):
                    u1, u2 = revblock.block_inverse(u1, u2, self._layers(b, 0), self._layers(b, 1),
                                                    self.eps, self.store)
            self.last_used = dict(u=(u1, u2), P=list(P))
            acts = []
            for b in range(self.blocks):
                acts.append((u1, u2))
                u1, u2 = revblock.block_forward(u1, u2, self._layers(b, 0, P),
                                                self._layers(b, 1, P), self.eps, self.store)
            for b in reversed(range(self.blocks)):
                r = revblock.block_vjp(acts[b][0], acts[b][1], g1, g2, self._layers(b, 0, P),
                                       self._layers(b, 1, P), self.eps, self.store)
                take(b, r)
                g1, g2 = r["dx1"], r["dx2"]
        if not self.front:
            # purely reversible stage: the input gradient is the blocks' one and
            # the stage sends back the block input it used (reconstructed)
            self.last_used["dx"] = np.concatenate([g1, g2], axis=-1)
            return self.last_used["dx"], grads
        # non-reversible front: recompute from the buffered input
        _, _, graph = self._front(x1, x2, P)
        stem = self.front == "stem"
        stride = 1 if stem else 2
        dx, (dw, dg, db) = nonrev_vjp(np.concatenate([g1, g2], axis=-1), self._w(0, P),
                                      P[1], graph, stride, relu=stem,
                                      store=self.store)
        grads[0:3] = [dw, dg, db]
        h = graph[1]
        self.run_mean[0], self.run_var[0] = bn.running_update(
            self.run_mean[0], self.run_var[0], graph[3], h.shape[0] * h.shape[1] * h.shape[2],
            self.bn_momentum)
        return dx, grads

    def accumulate(self, grads, k):
        for a, g in zip(self.accum, grads):
            a += g / k
        self.t += 1

    def update(self, lr, mu, wd, nesterov, k):
        if self.t == 0 or self.t % k != 0:
            return False
        for i, name in enumerate(self.names):
            wdp = wd if name.endswith("weight") else 0.0
            self.params[i], self.buf[i] = sgd.step(self.params[i], self.accum[i], self.buf[i],
                                                   lr, mu, wdp, nesterov)
            self.accum[i] = np.zeros_like(self.accum[i])
        return True


def split_params(names: Sequence[str], params: Sequence[np.ndarray], stages: int):
    out = [([], []) for _ in range(stages)]
    for nm, p in zip(names, params):
        j = int(nm.split(".")[0][1:])
        out[j][0].append(p)
        out[j][1].append(nm)
    return out


class PetraNet:
    """Tick-level simulation of the PETRA schedule over J stages."""

    def __init__(self, params, names, stages: int, blocks_per_stage: int, eps=1e-5,
                 bn_momentum=0.1, dtype=np.float64, weight_view=None, store=None,
                 use_inputs=False, use_params=False, split_fronts=False):
        """`stages` levels of the network (widths); with split_fronts every front
        layer (stem or downsampling) and every reversible block is a stage of
        its own, the last block also owning the head, as in the paper's
        per-layer splits (Table 6, App. B): J = levels x (1 + blocks), and a
        reversible stage below another one reconstructs from the reconstruction
        that stage sends back."""
        self.use_inputs, self.use_params = use_inputs, use_params
        self.record: Optional[dict] = None   # (stage, micro-batch) -> parameter gradients
        self.stages = []
        groups = split_params(names, params, stages)
        for lv, (ps, ns) in enumerate(groups):
            last = lv == stages - 1
            if not split_fronts:
                self.stages.append(NetStage(ps, ns, lv == 0, last, blocks_per_stage, eps,
                                            bn_momentum, dtype, weight_view, store))
                continue
            fr = [i for i, nm in enumerate(ns) if ".stem" in nm or ".trans" in nm]
            self.stages.append(NetStage([ps[i] for i in fr], [ns[i] for i in fr], lv == 0, False,
                                        0, eps, bn_momentum, dtype, weight_view, store,
                                        front="stem" if lv == 0 else "trans"))
            for b in range(blocks_per_stage):
                lb = last and b == blocks_per_stage - 1
                sel = [i for i, nm in enumerate(ns)
                       if f".b{b}." in nm or (lb and ".fc." in nm)]
                self.stages.append(NetStage([ps[i] for i in sel], [ns[i] for i in sel], False, lb,
                                            1, eps, bn_momentum, dtype, weight_view, store,
                                            front=None))
        self.J = len(self.stages)
        self.dtype = dtype
        self.fwd_msg: List[Optional[tuple]] = [None] * stages
        self.bwd_msg: List[Optional[tuple]] = [None] * stages
        self.trace: List[tuple] = []

    def fwd_batch(self, t: int, j: int) -> int:
        return t - j

    def bwd_batch(self, t: int, j: int) -> int:
        return t - (2 * self.J - 2 - j)

    def tick(self, t: int, images: Callable[[int], np.ndarray], labels: Callable[[int], np.ndarray],
             n_micro: int, lr: float, mu: float, wd: float, nesterov=True, k=1):
        """One tick of every stage; returns the loss computed this tick (or None)."""
        J = self.J
        new_fwd: List[Optional[tuple]] = [None] * J
        new_bwd: List[Optional[tuple]] = [None] * J
        loss = None
        did_bwd = [False] * J
        for j, st in enumerate(self.stages):
            m = self.fwd_batch(t, j)
            last_out = None
            if 0 <= m < n_micro:
                if j == 0:
                    x1, x2 = np.asarray(images(m), self.dtype), None
                else:
                    x1, x2 = self.fwd_msg[j - 1]
                    if st.front:
                        st.buffer[m] = (x1, x2)
                y1, y2 = st.forward(x1, x2, m)
                if st.last:
                    last_out = (y1, y2)
                else:
                    new_fwd[j] = (y1, y2)
            mb = self.bwd_batch(t, j)
            if 0 <= mb < n_micro:
                if st.last:
                    y1, y2 = last_out
                    lab = labels(mb)
                    loss, hc = head_loss(np.concatenate([y1, y2], -1), st.params[-2], st.params[-1], lab)
                    dx, dwfc, dbfc = head_vjp(st.params[-2], lab, hc)
                    c = y1.shape[-1]
                    g1, g2 = st.store(dx[..., :c]), st.store(dx[..., c:])
                else:
                    y1, y2, g1, g2 = self.bwd_msg[j + 1]
                if j == 0:
                    bx1, bx2 = np.asarray(images(mb), self.dtype), None
                elif st.front:
                    bx1, bx2 = st.buffer.pop(mb)
                else:
                    bx1 = bx2 = None
                dx, grads = st.backward(y1, y2, g1, g2, bx1, bx2, k, mb, self.use_inputs,
                                        self.use_params)
                if st.last:
                    grads[-2], grads[-1] = dwfc, dbfc
                if self.record is not None:
                    self.record[(j, mb)] = dict(grads=grads, y=(y1, y2), g=(g1, g2),
                                                x_in=(bx1, bx2), **st.last_used)
                st.accumulate(grads, k)
                did_bwd[j] = True
                if j > 0:
                    # a stage with a front sends back its buffered input, a
                    # reversible one the block input it used (reconstructed)
                    sx1, sx2 = (bx1, bx2) if st.front else st.last_used["u"]
                    c = sx1.shape[-1]
                    new_bwd[j] = (sx1, sx2, dx[..., :c], dx[..., c:])
            self.trace.append((t, j, m if 0 <= m < n_micro else None,
                               mb if 0 <= mb < n_micro else None))
        for j, st in enumerate(self.stages):
            if did_bwd[j]:
                st.update(lr, mu, wd, nesterov, k)
        self.fwd_msg, self.bwd_msg = new_fwd, new_bwd
        return loss

    def probe_tick(self, t: int, images, labels, n_micro: int, use_inputs: bool,
                   use_params: bool) -> Dict[str, np.ndarray]:
        """The parameter gradients (unscaled, by name) that the backward passes
        of tick t would produce in the given buffer variant, leaving this
        schedule untouched (App. B: the gradients compared at a snapshot).
        Stages without a backward at tick t give zeros."""
        c = copy.deepcopy(self)
        c.use_inputs, c.use_params = use_inputs, use_params
        c.record = {}
        c.tick(t, images, labels, n_micro, 0.0, 0.0, 0.0, True, 1 << 40)
        out = {}
        for j, st in enumerate(c.stages):
            got = [r["grads"] for (jj, _), r in c.record.items() if jj == j]
            for i, nm in enumerate(st.names):
                out[nm] = got[0][i] if got else np.zeros_like(st.params[i])
        return out

    def probe_backprop(self, images: np.ndarray, labels: np.ndarray) -> Dict[str, np.ndarray]:
        """End-to-end gradient (by name) of one micro-batch's loss at the
        current parameters of every stage, leaving this schedule untouched."""
        c = copy.deepcopy(self)
        for st in c.stages:
            st.accum = [np.zeros_like(p) for p in st.params]
        K = 1 << 40
        c.backprop_step(images, labels, 0.0, 0.0, 0.0, True, K)
        return {nm: a * K for st in c.stages for nm, a in zip(st.names, st.accum)}

    def backprop_step(self, images: np.ndarray, labels: np.ndarray, lr: float, mu: float,
                      wd: float, nesterov=True, k=1):
        """Reversible backpropagation of one micro-batch, the baseline of the
        iteration-time comparison (Sec. 4.2, Table 5): the forward of every
        stage in order, the loss, then the backward of every stage from the last
        to the first with the parameters the forward used (exact gradients),
        each stage accumulating and updating after its own backward.  The
        stages' front layers see their input as in the schedule (the previous
        stage's output); the blocks rebuild their inputs from their outputs."""
        ins = []
        x1, x2 = np.asarray(images, self.dtype), None
        for st in self.stages:
            ins.append((x1, x2))
            x1, x2 = st.forward(x1, x2)
        last = self.stages[-1]
        loss, hc = head_loss(np.concatenate([x1, x2], -1), last.params[-2], last.params[-1], labels)
        dx, dwfc, dbfc = head_vjp(last.params[-2], labels, hc)
        c = x1.shape[-1]
        y1, y2, g1, g2 = x1, x2, last.store(dx[..., :c]), last.store(dx[..., c:])
        for j in reversed(range(self.J)):
            st = self.stages[j]
            bx1, bx2 = ins[j]
            dx, grads = st.backward(y1, y2, g1, g2, bx1, bx2, k)
            if st.last:
                grads[-2], grads[-1] = dwfc, dbfc
            st.accumulate(grads, k)
            st.update(lr, mu, wd, nesterov, k)
            if j > 0:
                c = bx1.shape[-1]
                y1, y2, g1, g2 = bx1, bx2, dx[..., :c], dx[..., c:]
        return loss
