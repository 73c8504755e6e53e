"""Writes small_layer.json: oracle outputs for two small hand-specified layers
(a plain LSTM visited forward and an LSTMP visited in reverse).  Calls only
the oracle; the inputs are simple closed-form patterns, not random draws."""
import json
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))
import oracle  # noqa: E402


def pattern(shape, a, b):
    n = int(np.prod(shape))
    k = np.arange(n, dtype=np.float64)
    return (np.sin(a * k + b) * 0.5).reshape(shape)


def case(name, T, B, I, H, Hp, reverse):
    Hr = Hp if Hp else H
    inp = dict(x=pattern((T, B, I), 0.7, 0.1), W=pattern((4 * H, I), 1.3, 0.2),
               R=pattern((4 * H, Hr), 0.9, 0.3), b=pattern((4 * H,), 2.1, 0.4),
               P=pattern((Hp, H), 1.7, 0.5) if Hp else None,
               h0=pattern((B, Hr), 0.5, 0.6), c0=pattern((B, H), 0.3, 0.7),
               dy=pattern((T, B, Hr), 1.1, 0.8), dhT=pattern((B, Hr), 0.4, 0.9), dcT=pattern((B, H), 0.2, 1.0))
    o = oracle.layer_forward(inp["x"], inp["W"], inp["R"], inp["b"], inp["P"], inp["h0"], inp["c0"], reverse=reverse)
    g = oracle.layer_backward(inp["x"], inp["W"], inp["R"], inp["b"], inp["dy"], inp["P"], inp["h0"], inp["c0"],
                              inp["dhT"], inp["dcT"], reverse=reverse)
    exp = dict(o, **g)
    return dict(name=name, reverse=reverse,
                inputs={k: (None if v is None else v.tolist()) for k, v in inp.items()},
                expected={k: v.tolist() for k, v in exp.items()})


if __name__ == "__main__":
    cases = [case("lstm_T3_B2_I3_H2", 3, 2, 3, 2, 0, False), case("lstmp_rev_T3_B2_I2_H3_Hp2", 3, 2, 2, 3, 2, True)]
    with open(os.path.join(HERE, "small_layer.json"), "w") as f:
        json.dump(dict(source="tests/golden/make_golden.py (oracle only)", cases=cases), f, indent=1)
