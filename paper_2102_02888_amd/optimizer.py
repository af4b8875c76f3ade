"""Algorithm 1 end to end: Adam warm-up, variance freeze, compression stage.

OnebitAdam drives one State through the two stages of 1-bit Adam
(Algorithm 1): original Adam (eq. (alg:v)) for the warm-up steps, then, with
the variance frozen, error-compensated 1-bit compressed momentum steps.  The
warm-up ends after a fixed number of steps T_w, or, with a
VarianceFreezeDetector, at the step the detector picks (Section 7.1).  The
caller fills `grads` (one row per simulated worker) before each step().

With graph=True the steady compressed step (packed momentum, from the second
compression step on) is captured once in a HIP graph and replayed: one launch
instead of five, for models small enough that launch latency matters.  The
graph holds the state's buffer addresses, so `grads` must be filled in place;
it is captured again whenever lr, beta1 or eps changes.
"""
import torch

from .freeze import VarianceFreezeDetector
from .onebit import State


class OnebitAdam:
    def __init__(self, plan, device, lr, beta1=0.9, beta2=0.999, eps=1e-8, warmup_steps=None,
                 freeze=None, bias_correction=False, packed_momentum=True,
                 grad_dtype=torch.float32, graph=False):
        if (warmup_steps is None) == (freeze is None):
            raise ValueError("give exactly one of warmup_steps (fixed T_w) and freeze "
                             "(a VarianceFreezeDetector)")
        if freeze is not None and not isinstance(freeze, VarianceFreezeDetector):
            raise TypeError("freeze must be a VarianceFreezeDetector")
        self.state = State(plan, device, packed_momentum=packed_momentum, grad_dtype=grad_dtype)
        self.lr, self.beta1, self.beta2, self.eps = lr, beta1, beta2, eps
        self.warmup_steps = warmup_steps
        self.freeze = freeze
        self.bias_correction = bool(bias_correction)
        self.t = 0             # steps taken
        self.frozen_at = None  # last warm-up step, once the variance is frozen
        self.graph = bool(graph)
        self._graph = None     # captured compressed step and the arguments it holds
        self._graph_args = None

    @property
    def grads(self):
        return self.state.grads

    @property
    def x(self):
        return self.state.x

    @property
    def in_warmup(self):
        return self.frozen_at is None

    def step(self, lr=None, stream=None):
        """One step of Algorithm 1 on the gradients in `grads`; returns
        "warmup" or "compressed" for the kind of step taken.  With a freeze
        detector each warm-up step reads back one fp64 norm (a host sync)."""
        lr = self.lr if lr is None else lr
        self.t += 1
        if self.in_warmup:
            self.state.warmup(lr, self.beta1, self.beta2, self.eps, self.t,
                              bias_correction=int(self.bias_correction), stream=stream)
            if self.freeze is not None:
                done = self.freeze.update(self.t, self.state.variance_l1_norm(stream=stream))
            else:
                done = self.t >= self.warmup_steps
            if done:
                self.frozen_at = self.t
            return "warmup"
        self._compressed_step(lr, stream)
        return "compressed"

    def _compressed_step(self, lr, stream):
        st = self.state
        if not (self.graph and st.momentum_is_packed()):
            st.step(lr, self.beta1, self.eps, stream=stream)
            return
        args = (float(lr), float(self.beta1), float(self.eps))
        if self._graph is None or self._graph_args != args:
            g = torch.cuda.CUDAGraph()
            done = st.compression_steps
            with torch.cuda.graph(g):  # records the launches; nothing runs
                st.step(*args)
            st.compression_steps = done
            self._graph, self._graph_args = g, args
        if stream is None:
            self._graph.replay()
        else:
            with torch.cuda.stream(stream):
                self._graph.replay()
        st.compression_steps += 1

    def state_dict(self):
        sd = self.state.state_dict()
        sd["t"] = torch.tensor([self.t], dtype=torch.int64)
        sd["frozen_at"] = torch.tensor([-1 if self.frozen_at is None else self.frozen_at],
                                       dtype=torch.int64)
        return sd

    def load_state_dict(self, sd):
        """Restores a state_dict(); a freeze detector's norm history is not
        part of it, so a run resumed inside an auto-detected warm-up starts
        the detector afresh."""
        self.state.load_state_dict(sd)
        self._graph = self._graph_args = None
        self.t = int(sd["t"][0])
        f = int(sd["frozen_at"][0])
        self.frozen_at = None if f < 0 else f
