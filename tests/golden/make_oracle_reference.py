"""Writes tests/golden/oracle_reference_run.json: digests of the oracle's
state after a small seeded run (2 Adam warm-up steps, 3 compression steps).
It calls only oracle/ and synth/.  The test that reads it fails when the
oracle's arithmetic changes, so that such a change is made deliberately."""
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import synth  # noqa: E402

WORKLOAD = dict(name="golden", numel=[1000, 64, 0, 130, 5000], n=3, warmup_steps=2, steps=3)


def run():
    wl = synth.Workload(**WORKLOAD)
    L = oracle.Layout(wl.numel, wl.n)
    x = synth.host_params(wl, L.D)
    x[~L.real_mask()] = 0
    m = np.zeros(L.D, np.float32)
    v = np.zeros(L.D, np.float32)
    for t in range(1, wl.warmup_steps + 1):
        g = synth.host_grads(wl, L.D, L.tensor_off, t)
        oracle.warmup_step(L, x, m, v, g, wl.n, wl.lr, wl.beta1, wl.beta2, wl.eps, 0, t)
    st = oracle.State(L, x, m, v)
    for t in range(wl.warmup_steps + 1, wl.warmup_steps + wl.steps + 1):
        st.step(synth.host_grads(wl, L.D, L.tensor_off, t), wl.lr, wl.beta1, wl.eps)
    return {"x": st.x, "m": st.m, "v": st.v, "delta": st.delta, "delta_bar": st.delta_bar,
            "wbits": st.wbits, "sbits": st.sbits, "wscales": st.wscales, "sscales": st.sscales}


def digests(state):
    return {k: hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()
            for k, a in sorted(state.items())}


if __name__ == "__main__":
    out = {"workload": WORKLOAD, "sha256": digests(run())}
    path = os.path.join(HERE, "oracle_reference_run.json")
    json.dump(out, open(path, "w"), indent=1)
    print(path)
