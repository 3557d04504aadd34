"""Several virtual workers of one stage, simulated on one GPU under WSP.

Each minibatch runs through the C ABI: hp_wsp_weights (the ring version with
the local updates 1..q-W, HetPipe Sec. 4), hp_stage_forward and
hp_stage_backward at those weights, hp_wsp_local_update (u = -lr g, or with
momentum u = -lr v, v = mu v + g; ring write, wave accumulation; lr may
change per minibatch, e.g. the sigma/sqrt(t) schedule of Theorem 1), and at a wave end hp_wsp_push_wave followed by
hp_wsp_pull, the clock-distance gate of Sec. 5 -- by default the three at a
wave end as one call, hp_wsp_wave_end (bit-identical results).  A VW whose pull reports
HP_WOULD_BLOCK stops until another VW's push lets its pull succeed.

Scheduling (the paper leaves it open; virtual workers are independent
machines): VW n completes a minibatch every T_n time units; the runnable VW
with the smallest (next completion time, id) goes next; a VW unblocked at
time t resumes at max(its next completion time, t); minibatches already in
flight in a blocked VW do not complete until it is unblocked.

Every minibatch, push, pull and block is recorded in ``events``:
  ("mb", n, q, V)  ("push", n, c, c_g)  ("pull", n, g)  ("block", n, need)
where V is the version vector of the weights minibatch q used.
"""
from __future__ import annotations

import torch

from .hetpipe import ParameterServer, Stage, VirtualWorker


class Deadlock(RuntimeError):
    pass


class WSPDriver:
    def __init__(self, stage: Stage, w0: torch.Tensor, N: int, s_local: int, D: int, lr,
                 data_fn, periods=None, stream=None, need_dx=False, on_minibatch=None,
                 grad_fn=None, P=None, momentum=0.0, fused=True):
        # grad_fn(n, q, w_ptr, grad): fill `grad` without a stage (WSP-only runs)
        self.stage = stage
        self.grad_fn = grad_fn
        # lr: a step size, or a function lr(n, q) of the VW and its minibatch
        self.N, self.W, self.D = N, s_local + 1, D
        self.lr = lr if callable(lr) else (lambda n, q, _lr=lr: _lr)
        self.data_fn = data_fn
        self.T = list(periods) if periods else [1] * N
        self.P = stage.P if stage is not None else P
        self.ps = ParameterServer(self.P, w0, N, D, stream)
        self.vws = [VirtualWorker(self.ps, n, s_local) for n in range(N)]
        if momentum:
            for v in self.vws:
                v.set_momentum(momentum)
        dev = w0.device
        self.grad = torch.empty(max(self.P, 1), dtype=torch.float32, device=dev)
        self.loss = torch.empty(1, dtype=torch.float32, device=dev)
        self.y = self.dx = None
        if stage is not None:
            H, W, C = stage.output_shape(-1)
            self.y = torch.empty((stage.batch, H, W, C), dtype=torch.float32, device=dev)
            if need_dx:
                self.dx = torch.empty((stage.batch, stage.H, stage.W, stage.C),
                                      dtype=torch.float32, device=dev)
        self.t = list(self.T)
        self.blocked = [False] * N
        self.done = [0] * N
        self.events = []
        self.on_minibatch = on_minibatch
        # a wave's last minibatch: local update + push + gate in one call
        # (hp_wsp_wave_end), or the three calls in turn
        self.fused = fused

    def close(self):
        for v in self.vws:
            v.close()
        self.ps.close()

    # ------------------------------------------------------------------
    def minibatch(self, n):
        vw = self.vws[n]
        q = vw.state()["p"] + 1
        self.events.append(("mb", n, q, vw.version()))
        w = vw.weights()
        if self.grad_fn is not None:
            self.grad_fn(n, q, w, self.grad)
        elif self.stage.has_loss:
            x, labels, _ = self.data_fn(n, q)
            self.stage.forward(w, x, self.y, labels, self.loss)
            self.stage.backward(w, None, self.dx, self.grad)
        else:
            x, _, dy = self.data_fn(n, q)
            self.stage.forward(w, x, self.y)
            self.stage.backward(w, dy, self.dx, self.grad)
        if self.on_minibatch is not None:
            self.on_minibatch(n, q, self)
        if q % self.W == 0 and self.fused:
            self._push_and_gate(n, self.lr(n, q))
        else:
            vw.local_update(self.grad, self.lr(n, q))
            if q % self.W == 0:
                self._push_and_gate(n)
        self.t[n] += self.T[n]
        self.done[n] = q

    def _pulled(self, m):
        s = self.vws[m].state()
        self.events.append(("pull", m, s["g"]))

    def _push_and_gate(self, n, lr=None):
        """Push of VW n's completed wave and its gate; with lr given, the wave's
        last local update, the push and the gate in one call (hp_wsp_wave_end)."""
        vw = self.vws[n]
        g0 = vw.state()["g"]
        if lr is not None:
            ok = vw.wave_end(self.grad, lr)
        else:
            vw.push_wave()
        s = vw.state()
        self.events.append(("push", n, s["c"], self.ps.clock()))
        if lr is None:
            ok = vw.pull()
        if ok:
            if vw.state()["g"] != g0:
                self._pulled(n)
        else:
            self.blocked[n] = True
            self.events.append(("block", n, s["c"] - self.D))
        now = self.t[n]
        for m in range(self.N):
            if self.blocked[m] and self.vws[m].pull():
                self.blocked[m] = False
                self._pulled(m)
                self.t[m] = max(self.t[m], now)

    def run(self, waves, max_minibatches=None):
        target = waves * self.W
        count = 0
        while True:
            cand = [n for n in range(self.N) if not self.blocked[n] and self.done[n] < target]
            if not cand:
                if any(self.blocked):
                    raise Deadlock("no runnable virtual worker; blocked: %s"
                                   % [n for n in range(self.N) if self.blocked[n]])
                break
            n = min(cand, key=lambda m: (self.t[m], m))
            self.minibatch(n)
            count += 1
            if max_minibatches is not None and count >= max_minibatches:
                break
        return self.events
