"""Phase-aware activation precision policy (oracle; test infrastructure).

Algorithm 1 step 2: b_x = 8 for a layer in the sensitive set S, else 4; weights
and KV caches stay at 4 bits (step 1).  Eq. 21 instantiates S = {1, 2, 3, L}
with layers indexed from 1; the efficiency study (Section 4.9) lists the same
set 0-indexed as {0, 1, 2, L-1}.  This module works 0-indexed.

An explicit mask (nonzero = 8-bit) overrides the default set, for sets chosen
by the Eq. 20 rule or by a seeded draw.
"""

__all__ = ["layer_policy_ref", "default_sensitive_set"]


def default_sensitive_set(num_layers):
    """Eq. 21, 0-indexed: {0, 1, 2, L-1} intersected with the valid layers."""
    L = int(num_layers)
    if L < 1:
        raise ValueError("num_layers must be >= 1")
    return sorted({i for i in (0, 1, 2, L - 1) if 0 <= i < L})


def layer_policy_ref(num_layers, mask=None):
    """bits[l] in {4, 8} for l = 0 .. L-1."""
    L = int(num_layers)
    if L < 1:
        raise ValueError("num_layers must be >= 1")
    if mask is None:
        sens = set(default_sensitive_set(L))
    else:
        mask = list(mask)
        if len(mask) != L:
            raise ValueError("mask length must equal num_layers")
        sens = {i for i, v in enumerate(mask) if v}
    return [8 if i in sens else 4 for i in range(L)]
