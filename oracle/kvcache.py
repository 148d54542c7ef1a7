"""Oracle: the KV cache of an L-Layer after absorption (test infrastructure).

Sec. 3.1 step 3 and Sec. 3.3: a layer turned into an L-Layer permanently
evicts its history and from then on attends only to its local context, the
sink prefix plus the most recent keys (Sec. 3.4, Eq. 7). The oracle states
WHAT such a layer holds, not how it is stored: after every chunk it holds the
local set of the whole key sequence generated so far.

Reading: the local set keeps its definition of Eq. 7
forever, with the sink taken from the first keys of the sequence and the
window from its last ``window`` keys; keys are rows of the hidden layout
[keys, H * d].
"""

import numpy as np

from .attention import visible_key_sets


def evict_local(k, v, cache_len, window, sink_len=0):
    """Rows of the local set of a cache of ``cache_len`` keys (Eq. 7):
    the sink rows, then the window rows, each in cache order."""
    local, _ = visible_key_sets(int(cache_len), int(window), int(sink_len))
    k = np.asarray(k)[: int(cache_len)]
    v = np.asarray(v)[: int(cache_len)]
    return k[local], v[local]


class LocalHistory:
    """Key/value rows an L-Layer holds as chunks keep arriving: the local set
    of everything appended so far (a plain list of all rows; slow and
    obviously correct)."""

    def __init__(self, k, v, cache_len, window, sink_len=0):
        self.k = [np.asarray(k)[: int(cache_len)]]
        self.v = [np.asarray(v)[: int(cache_len)]]
        self.window = int(window)
        self.sink = int(sink_len)

    def append(self, k_new, v_new):
        self.k.append(np.asarray(k_new))
        self.v.append(np.asarray(v_new))

    def rows(self):
        k = np.concatenate(self.k, axis=0)
        v = np.concatenate(self.v, axis=0)
        return evict_local(k, v, k.shape[0], self.window, self.sink)
