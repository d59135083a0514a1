"""Token-level model of asynchronous state reconciliation (Algorithm 1).

TEST INFRASTRUCTURE ONLY (like the rest of ``oracle/``): the tests compare the
GPU driver's bookkeeping with this model; nothing on the product path imports
it.  It computes no attention: it tracks which token ids each cache holds and
which ids every served task computes, following Algorithm 1 step by step.

Vocabulary (paper Sec. III-D and Algorithm 1):
* ``X_pre``: the fixed state prefix; ``X_chunks``: state chunks appended one
  per task; ``X_static = X_pre (+) X_chunks``.
* ``Evict``: the rule of the paper's robot runs (Sec. IV), which discards the
  oldest half of the chunks and keeps the prefix.
* Increment(dX): X_static <- X_static (+) dX; while a reconciliation runs the
  chunk is also buffered; at |X_static| >= tau_mem a reconciliation starts:
  X_E <- Evict(X_static), warm-up of X_E on the secondary resource.
* Reconcile: after the warm-up, while the buffer holds more than N_catchup
  tokens, absorb it into X_E and extend the secondary cache; then swap the
  resources.  Chunks still buffered at the swap are computed by the next task
  on the new primary (Algorithm 1's note on the remainder).

Asynchrony is an input: the caller says when the secondary's outstanding work
has finished (``secondary_done``), so the model follows any interleaving.
Token ids are plain integers; a chunk is a list of ids.
"""
from __future__ import annotations


def flat(chunks) -> list:
    return [t for c in chunks for t in c]


def evict_oldest_half(chunks: list) -> list:
    """The robot runs' rule: drop the oldest half (rounded down) of the chunks."""
    return [list(c) for c in chunks[len(chunks) // 2:]]


class AsrModel:
    def __init__(self, x_pre, tau_mem: int, n_catchup: int):
        self.x_pre = list(x_pre)
        self.chunks: list = []            # X_chunks of the primary's logical state
        self.static_len = len(self.x_pre)  # |X_static|
        self.tau_mem = tau_mem
        self.n_catchup = n_catchup        # tokens
        self.reconciling = False
        self.buffer: list = []            # Delta X_buffer, as chunks
        self.x_e_chunks: list = []        # chunks of X_E (after X_pre)
        self.primary_cached: list = list(x_pre)   # ids in the primary's cache, in order
        self.primary_pending: list = []   # ids the primary's next task must still compute
        self.secondary_busy = False       # warm-up or a catch-up not yet finished
        self.phase = "idle"               # idle | warmup | catchup
        self.swaps = 0
        self.evictions = 0
        self.log: list = []

    def x_static(self) -> list:
        return self.x_pre + flat(self.chunks)

    def x_e(self) -> list:
        return self.x_pre + flat(self.x_e_chunks)

    # -- Algorithm 1, procedure Increment -------------------------------------
    def increment(self, chunk) -> list:
        """Append one state chunk and serve one task on the primary; returns the
        ids the task computes (its cached prefix excluded), in order."""
        chunk = list(chunk)
        self.chunks.append(chunk)
        self.static_len += len(chunk)
        if self.reconciling:
            self.buffer.append(chunk)
        if self.static_len >= self.tau_mem and not self.reconciling:
            self.x_e_chunks = evict_oldest_half(self.chunks)
            self.reconciling = True
            self.secondary_busy = True
            self.phase = "warmup"
            self.evictions += 1
            self.log.append(("warmup", len(self.x_e())))
        computed = self.primary_pending + chunk
        self.primary_cached += computed
        self.primary_pending = []
        return computed

    # -- Algorithm 1, procedure Reconcile (advanced when work completes) ---------
    def secondary_done(self) -> None:
        """The secondary's outstanding warm-up or catch-up has finished."""
        assert self.secondary_busy
        self.secondary_busy = False
        if len(flat(self.buffer)) > self.n_catchup:
            self.log.append(("catchup", len(flat(self.buffer))))
            self.x_e_chunks += self.buffer
            self.buffer = []
            self.secondary_busy = True
            self.phase = "catchup"
            return
        # Swap: the secondary becomes the primary.  Its logical state is
        # X_E (+) remainder; the remainder is computed by its next task.
        remainder = self.buffer
        self.buffer = []
        self.chunks = [list(c) for c in self.x_e_chunks] + [list(c) for c in remainder]
        self.static_len = len(self.x_pre) + sum(len(c) for c in self.chunks)
        self.primary_cached = self.x_e()
        self.primary_pending = flat(remainder)
        self.reconciling = False
        self.phase = "idle"
        self.swaps += 1
        self.log.append(("swap", len(flat(remainder))))
