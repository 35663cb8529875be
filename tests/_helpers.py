"""Shared helpers for the parity tests: oracle references and error metrics."""
import sys

import numpy as np

import oracle

TOL = {"f32": 1e-5, "bf16": 2e-2}
KEYS = ("y", "hT", "cT", "dx", "dW", "dbias", "dh0", "dc0")


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def oracle_reference(inp, layers, dtype, cell="lstm", ponder_max=4):
    """fp64 oracle (bf16-emulating for bf16 workloads) of the full fwd + bwd.
    For the RNN and GRU cells, cT and dc0 are zeros (the library writes zeros
    there)."""
    precision = "bf16" if dtype == "bf16" else "fp64"
    if cell in ("rnn", "gru"):
        fwd, bwd = ((oracle.stacked_rnn_forward, oracle.stacked_rnn_backward) if cell == "rnn"
                    else (oracle.stacked_gru_forward, oracle.stacked_gru_backward))
        x = inp["x"].astype(np.float64)
        Ws = [w.astype(np.float64) for w in inp["W"]]
        bs = [b.astype(np.float64) for b in inp["bias"]]
        h0 = inp["h0"].astype(np.float64)
        dy = None if inp["dy"] is None else inp["dy"].astype(np.float64)
        y, hT, tapes = fwd(x, inp["seq_len"], Ws, bs, h0, precision)
        g = bwd(tapes, dy, inp["dhT"].astype(np.float64))
        return dict(y=y, hT=hT, cT=np.zeros_like(hT), dx=g["dx"], dW=g["dW"], dbias=g["dbias"],
                    dh0=g["dh0"], dc0=np.zeros_like(hT), T_eff=tapes[0]["T_eff"])
    x = inp["x"].astype(np.float64)
    Ws = [w.astype(np.float64) for w in inp["W"]]
    bs = [b.astype(np.float64) for b in inp["bias"]]
    h0 = inp["h0"].astype(np.float64)
    c0 = inp["c0"].astype(np.float64)
    dy = None if inp["dy"] is None else inp["dy"].astype(np.float64)
    if cell == "act":
        y, hT, cT, tapes = oracle.stacked_act_forward(x, inp["seq_len"], Ws, bs, h0, c0, precision,
                                                      ponder_max)
        g = oracle.stacked_act_backward(tapes, dy, inp["dhT"].astype(np.float64),
                                        inp["dcT"].astype(np.float64))
        return dict(y=y, hT=hT, cT=cT, dx=g["dx"], dW=g["dW"], dbias=g["dbias"], dh0=g["dh0"],
                    dc0=g["dc0"], T_eff=tapes[0]["T_eff"], trips=[t["trips"] for t in tapes],
                    min_margin=min(t["min_margin"] for t in tapes))
    fwd, bwd = ((oracle.stacked_skip_forward, oracle.stacked_skip_backward) if cell == "skip"
                else (oracle.stacked_forward, oracle.stacked_backward))
    y, hT, cT, tapes = fwd(x, inp["seq_len"], Ws, bs, h0, c0, precision)
    g = bwd(tapes, dy, inp["dhT"].astype(np.float64), inp["dcT"].astype(np.float64))
    out = dict(y=y, hT=hT, cT=cT, dx=g["dx"], dW=g["dW"], dbias=g["dbias"],
               dh0=g["dh0"], dc0=g["dc0"], T_eff=tapes[0]["T_eff"])
    if cell == "skip":
        out["guards"] = [t["guards"] for t in tapes]
        out["margin"] = [t["margin"] for t in tapes]
        out["min_margin"] = min(t["min_margin"] for t in tapes)
    return out


def rel_err(got, ref):
    """max |got - ref| / max |ref| (absolute error when ref is all zero)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if not np.isfinite(got).all():
        return np.inf
    scale = np.abs(ref).max() if ref.size else 0.0
    err = np.abs(got - ref).max() if ref.size else 0.0
    return err / scale if scale > 0 else err


def compare(gpu, ref, tol, keys=KEYS, skip=()):
    errs = {}
    for k in keys:
        if k in skip:
            continue
        g, r = gpu[k], ref[k]
        if isinstance(r, list):
            errs[k] = max(rel_err(a, b) for a, b in zip(g, r))
        else:
            errs[k] = rel_err(g, r)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    return errs, bad
