"""Oracle for greedy target-only acceptance (test infrastructure only).

Sec. 3.2: acceptance is sequential, so keeping the first n_i drafts advances
1 + min(L_i, n_i) tokens (the bonus always counts).  Under greedy target-only
verification (Sec. 4.1 setup; App. A correctness) draft z_{i,j} is accepted
when it equals the target's argmax at the previous block position and every
earlier draft was accepted; the committed next token is the target's argmax
after the last accepted position.
"""
from __future__ import annotations

from typing import Dict

import numpy as np


def accept(draft: np.ndarray, keep_len: np.ndarray, cu: np.ndarray,
           argmax: np.ndarray) -> Dict[str, np.ndarray]:
    """a_i = largest m <= n_i with z_{i,j} == g[cu_i + j - 1] for all 1 <= j <= m;
    next_i = g[cu_i + a_i]; total = sum_i (a_i + 1)."""
    B = draft.shape[0]
    acc = np.zeros(B, dtype=np.int32)
    nxt = np.zeros(B, dtype=np.int32)
    for i in range(B):
        n = int(keep_len[i]) - 1
        a = 0
        while a < n and int(draft[i, a + 1]) == int(argmax[cu[i] + a]):
            a += 1
        acc[i] = a
        nxt[i] = argmax[cu[i] + a]
    total = np.array([int((acc.astype(np.int64) + 1).sum())], dtype=np.int32)
    return dict(accept_len=acc, next_tok=nxt, total=total)
