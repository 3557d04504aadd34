"""Wave Synchronous Parallel (WSP): the oracle's step-by-step simulation.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Follows HetPipe Sec. 4 (local staleness inside a virtual worker) and Sec. 5
(waves, clocks, the parameter server and the clock-distance bound D), in the
paper's order and notation:

  * s_local = N_m - 1; a wave is W = s_local + 1 minibatches.  Minibatches are
    numbered from 1, waves from 0; wave c holds minibatches c*W+1 .. (c+1)*W.
  * w_1 = ... = w_W = w_0 (the first W minibatches start from the initial
    weights); minibatch p uses the version that holds the local updates
    1 .. p-W (Sec. 4).  The W live versions sit in a ring: minibatch q reads
    slot (q-1) mod W, and when q completes the newest version plus u_q is
    written into that same slot, where minibatch q+W will read it.
  * local update w_local = w_local + u_p with u_p = -lr * gradient (Sec. 4; no
    1/(s_local+1) factor); the wave aggregate u~ is the sum of the wave's u_p.
  * at the end of wave c the VW pushes u~; the server applies w_g = w_g + u~
    (a sum over VWs, no averaging) and keeps c_g = min over VWs of the local
    clocks (Sec. 5, "Workings of WSP").
  * clock-distance bound: after finishing wave c (local clock c+1) the VW
    needs weights holding every VW's waves 0 .. c-D, i.e. a pulled global
    clock g >= c+1-D.  If its last pull already satisfies that it does not
    query the server at all (so the first D+1 waves run without a pull);
    otherwise it pulls w_g as soon as c_g >= c+1-D, and until then it is
    blocked (Sec. 5, "Global Staleness Bound").

Readings where the paper is silent (each listed in the design notes):
  * the pull replaces the local weights by w_g; since a pull directly follows
    the VW's own push, w_g already holds all of the VW's updates;
  * minibatches already in flight do not complete while their VW is blocked
    (so a VW includes exactly, not "at least", the updates the rules name);
  * several VWs are simulated by a discrete-event schedule: VW n completes a
    minibatch every T_n time units; the runnable VW with the smallest
    (next completion time, id) goes next; a VW unblocked at time t resumes at
    max(its next completion time, t).

Vector arithmetic is IEEE binary32 with round-to-nearest-even, one operation
at a time (no fused multiply-add):  u = (-lr) * g,  new = newest + u,
u~ = u (first minibatch of a wave) or u~ + u,  w_g = w_g + u~.

Optimizer variants (beyond the paper's plain SGD step):
  * ``lr`` may be a function lr(n, q) giving the step size of minibatch q of
    VW n, e.g. the eta_t = sigma / sqrt(t) schedule of Theorem 1 (see
    ``theorem1_schedule``);
  * ``momentum`` mu != 0 keeps a velocity per VW, updated at every local
    update before the step (heavy ball, no dampening):  v = mu * v + g,
    u = (-lr) * v; the velocity is local to the VW and is never pushed.

Every minibatch, push, pull and block is appended to ``events``:
  ("mb", n, q, V)        V = version vector of w_q: updates of each VW in it
  ("push", n, c, c_g)    local clock after the push and the new global clock
  ("pull", n, g)         pulled global clock
  ("block", n, need)
"""
from __future__ import annotations

import numpy as np


class DeadlockError(RuntimeError):
    pass


class WSP:
    def __init__(self, w0, N: int, s_local: int, D: int, lr, grad_fn,
                 periods=None, dtype=np.float32, record=False, momentum=0.0):
        self.N = N
        self.W = s_local + 1
        self.s_local = s_local
        self.D = D
        self.dtype = dtype
        self.lr = lr if callable(lr) else (lambda n, q, _lr=lr: _lr)
        self.mu = dtype(momentum) if dtype is not object else momentum
        self.grad_fn = grad_fn
        self.T = list(periods) if periods is not None else [1] * N
        assert len(self.T) == N
        w0 = np.asarray(w0, dtype=dtype)
        W = self.W
        # per-VW state
        self.ring = [[w0.copy() for _ in range(W)] for _ in range(N)]
        self.VR = [[[0] * N for _ in range(W)] for _ in range(N)]
        self.ut = [np.zeros_like(w0) for _ in range(N)]
        self.vel = [np.zeros_like(w0) for _ in range(N)]
        self.p = [0] * N          # minibatches completed
        self.c = [0] * N          # local clock = waves completed
        self.g = [0] * N          # global clock of the last pull
        self.t = list(self.T)     # next completion time
        self.blocked = [False] * N
        # parameter server
        self.wg = w0.copy()
        self.pushed = [0] * N     # waves of each VW contained in w_g
        self.cg = 0
        self.events = []
        self.record = record
        self.pushes = []          # (n, wave, u~) when record is set
        self.updates = {}         # (n, q) -> u_q when record is set

    # ------------------------------------------------------------------
    def _vec_add(self, a, b):
        return a + b

    def _pull(self, n):
        q = self.p[n]
        slot = (q - 1) % self.W
        self.ring[n][slot] = self.wg.copy()
        self.VR[n][slot] = [self.W * k for k in self.pushed]
        self.g[n] = self.cg
        self.events.append(("pull", n, self.g[n]))

    def _minibatch(self, n, now):
        W = self.W
        q = self.p[n] + 1
        slot = (q - 1) % W
        newest = (q - 2) % W
        w_q = self.ring[n][slot]
        self.events.append(("mb", n, q, tuple(self.VR[n][slot])))
        grad = np.asarray(self.grad_fn(n, q, w_q), dtype=self.dtype)
        lr = self.lr(n, q)
        neg_lr = -self.dtype(lr) if self.dtype is not object else -lr
        if self.mu != 0:
            self.vel[n] = self._vec_add(self.mu * self.vel[n], grad)
            u = neg_lr * self.vel[n]
        else:
            u = neg_lr * grad
        new = self._vec_add(self.ring[n][newest], u)
        vnew = list(self.VR[n][newest])
        vnew[n] += 1
        if (q - 1) % W == 0:
            self.ut[n] = u.copy()
        else:
            self.ut[n] = self._vec_add(self.ut[n], u)
        if self.record:
            self.updates[(n, q)] = u.copy()
        self.p[n] = q
        self.ring[n][slot] = new
        self.VR[n][slot] = vnew
        if q % W == 0:
            self._push_and_gate(n, q, now)
        self.t[n] += self.T[n]

    def _push_and_gate(self, n, q, now):
        cw = q // self.W - 1
        if self.record:
            self.pushes.append((n, cw, self.ut[n].copy()))
        self.wg = self._vec_add(self.wg, self.ut[n])
        self.pushed[n] += 1
        self.c[n] = cw + 1
        self.cg = min(self.c)
        self.events.append(("push", n, self.c[n], self.cg))
        need = self.c[n] - self.D
        if self.g[n] < need:
            if self.cg >= need:
                self._pull(n)
            else:
                self.blocked[n] = True
                self.events.append(("block", n, need))
        for m in range(self.N):
            if self.blocked[m] and self.c[m] - self.D <= self.cg:
                self.blocked[m] = False
                self._pull(m)
                self.t[m] = max(self.t[m], now)

    # ------------------------------------------------------------------
    def run(self, waves: int, stop_vw=None, stop_after=None):
        """Run until every VW completed ``waves`` waves.

        ``stop_vw``/``stop_after``: VW ``stop_vw`` stops for good after that
        many minibatches (a failed worker); the run then ends when no VW can
        proceed, raising DeadlockError if some VW is still blocked."""
        target = waves * self.W
        while True:
            cand = [n for n in range(self.N)
                    if not self.blocked[n] and self.p[n] < target
                    and not (n == stop_vw and self.p[n] >= stop_after)]
            if not cand:
                if any(self.blocked):
                    raise DeadlockError(
                        "no runnable virtual worker; blocked: %s"
                        % [n for n in range(self.N) if self.blocked[n]])
                break
            n = min(cand, key=lambda m: (self.t[m], m))
            self._minibatch(n, self.t[n])
        return self.events


def theorem1_schedule(sigma: float, N: int):
    """eta_t = sigma / sqrt(t) of Theorem 1 as a step-size function lr(n, q).
    The theorem numbers the updates of all VWs in one sequence that takes the
    VWs in turn: minibatch q of VW n is update t = (q - 1) * N + n + 1."""
    def lr(n, q):
        return sigma / np.sqrt((q - 1) * N + n + 1)
    return lr


def s_global(D: int, s_local: int) -> int:
    """Global staleness bound of Sec. 5: (D+1)(s_local+1) + s_local - 1."""
    return (D + 1) * (s_local + 1) + s_local - 1
