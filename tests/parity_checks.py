"""Shared checks of GPU outputs against the oracle (sampled positions, O6 metrics, rounding bound)."""
import sys

import numpy as np

import oracle as O


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def edge_samples(spec, rng, n_tok=64, n_ch=48):
    """Sampled output positions: first and last token and channel, the image
    border pixels of the first and last image, token and channel tile edges,
    then random positions."""
    T, C = spec.tokens, spec.C_out
    tok = [0, T - 1]
    if spec.conv is not None:
        OH, OW = spec.conv.OH, spec.conv.OW
        for b in (0, spec.n - 1):
            for oh, ow in ((0, 0), (0, OW - 1), (OH - 1, 0), (OH - 1, OW - 1), (0, OW // 2), (OH // 2, 0),
                           (OH - 1, OW // 2), (OH // 2, OW - 1)):
                tok.append((b * OH + oh) * OW + ow)
    for e in (32, 64, 128, 256):
        for t in (e - 1, e, T - e, T - e - 1):
            tok.append(t)
    ch = [0, C - 1]
    for e in (32, 64, 96, 128, 192, 256):
        ch += [e - 1, e, C - e]
    tok = sorted(set(t for t in tok if 0 <= t < T))
    ch = sorted(set(c for c in ch if 0 <= c < C))
    while len(tok) < min(n_tok, T):
        tok = sorted(set(tok) | {int(rng.integers(0, T))})
    while len(ch) < min(n_ch, C):
        ch = sorted(set(ch) | {int(rng.integers(0, C))})
    return np.array(tok), np.array(ch)


def sampled_outputs(spec, y, tok, ch):
    if spec.conv is None:
        return y[np.ix_(tok, ch)]
    flat = y.transpose(0, 2, 3, 1).reshape(spec.tokens, spec.C_out)
    return flat[np.ix_(tok, ch)]


def check_against_oracle(spec, inp, got, tok, ch, path, tol):
    """The GPU outputs at (tok, ch) against the oracle: infinity-norm and RMS
    relative errors within ``tol``, and every element within its rounding bound."""
    ref = O.forward_sampled(spec, inp, tok, ch)
    a_ref = O.forward_sampled(spec, O.abs_inputs(spec, inp), tok, ch)
    bound = O.rounding_bound(spec, ref, a_ref, path)
    e_inf, e_rms, e_el = O.rel_err_inf(got, ref), O.rel_err_rms(got, ref), O.rel_err_elem(got, ref)
    over = np.argwhere(np.abs(got - ref) > bound)
    _say(f"  inf={e_inf:.2e} rms={e_rms:.2e} elem(floor 1e-3 rms)={e_el:.2e} over_bound={len(over)}")
    for i, j in over[:5]:
        _say(f"    token {tok[i]} channel {ch[j]}: got {got[i, j]!r} ref {ref[i, j]!r} bound {bound[i, j]:.3e}")
    assert e_inf <= tol and e_rms <= tol
    assert len(over) == 0
