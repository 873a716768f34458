"""Speculative verification windows over the expert-slot cache (oracle; test infrastructure only).

The paper's Throughput Model section adds, for speculative decoding, an
extra-materialisation term: a verification step runs the target model on a
window of tokens (the last accepted token plus the draft's lookahead), and
that window can route to a wider union of experts than one decode step.  Its
speculative addendum measures the effect with a draft horizon of 4.

There is no draft model here.  A window is 1 + horizon consecutive positions
of the hidden-state stream; whether each draft token would pass verification
is an input (a boolean per step and draft position, drawn by the seeded
generator).  Per step, the standard acceptance rule: the accepted drafts are
the longest passing prefix; the step yields those tokens plus the target's
own next token, and the next window starts right after them.

With no attention between positions in this layer stack, a window's layer
call is the plain MoE layer applied to each of its tokens; the cache sees one
lookup per distinct routed expert of the whole window (the union over its
tokens), exactly as for any multi-token layer call.
"""
import numpy as np


def schedule(n_tokens, horizon, accept):
    """Verification steps generating n_tokens tokens.

    accept: [>= steps, horizon] bool, draft j of step s passes.  Returns a list of
    (start, accepted, generated) per step: the window covers positions
    start .. start + horizon; accepted = leading passes (0..horizon); generated =
    accepted + 1, cut at the last step so that the total is n_tokens."""
    out, t, s = [], 0, 0
    while t < n_tokens:
        a = 0
        while a < horizon and accept[s, a]:
            a += 1
        g = min(a + 1, n_tokens - t)
        out.append((t, a, g))
        t += g
        s += 1
    return out


def window_union(idx_window):
    """Distinct experts routed by any token of a window's layer call, ascending."""
    return np.unique(np.asarray(idx_window).ravel())
