"""Task Scheduler (Algorithms 2 and 3) with activation flow control
(Sec. 3.4.1) and the version bookkeeping of Algorithm 4.

Test infrastructure (see package docstring).  Readings taken where the
paper is silent:

* put() (Alg. 2) appends a model message to the model FIFO and an
  activation batch to the sending device's FIFO, subject to flow control.
* get() (Alg. 3) serves a pending model first (FIFO).  Otherwise it takes
  the device with the smallest consumption counter c_k among devices whose
  queue is not empty (an empty queue cannot be served), lowest index on
  ties, pops that device's oldest batch and increments c_k at the pick.
* Flow control: each device has a Sender Status, initially on.  A batch
  arriving while the status is off is dropped at the source.  An admitted
  batch switches the status off; after every enqueue to or dequeue from
  device k's queue, the status of k is switched back on if the total number
  of queued batches is below the cap omega.
* Memory: the pool has n_slots batch slots; omega = n_slots - K so that
  the at most one in-flight batch per device plus the batch in service
  always fit (queued <= omega + K - 1, plus one in service).  Free slots
  form a stack that starts as 0, 1, 2, ... (lowest id first); a released
  slot goes on top.
* Aggregation versions (Alg. 4): staleness s = t - t_k; a model with
  s > D is skipped and t is unchanged; otherwise t increases by one.
* FIFO policy (the scheduler ablation of Sec. 6.5): get() serves the
  activation batch admitted earliest over all devices instead of the
  least-served device; c_k is still counted.
* 'Turn-on' signals (Sec. 3.4.1): a signal is counted each time the check
  after an enqueue or dequeue switches an off Sender back on.
* Leaving and rejoining (Sec. 3.4.2, dropout of Sec. 6.4): a device that
  leaves has its Sender switched off and kept off (it sends nothing); the
  batches it already sent stay queued and are served as usual.  A device
  that rejoins starts with its Sender on, like a device joining for the
  first time, and keeps its counter c_k.
"""
from __future__ import annotations

from collections import deque


class TaskScheduler:
    def __init__(self, K: int, n_slots: int | None = None, policy: str = "counter"):
        if policy not in ("counter", "fifo"):
            raise ValueError(policy)
        self.policy = policy
        self.K = K
        self.n_slots = n_slots
        self.omega = None if n_slots is None else n_slots - K
        if self.omega is not None and self.omega < 1:
            raise ValueError("pool too small for the number of devices")
        self.q_model = deque()
        self.q_act = [deque() for _ in range(K)]
        self.c = [0] * K
        self.sender_on = [True] * K
        self.seq = [0] * K
        self.free = None if n_slots is None else list(range(n_slots - 1, -1, -1))
        self.in_service = None
        self.t = 0
        self.refused = 0
        self.peak_queued = 0
        self.active = [True] * K
        self.admissions = 0  # admission order over all devices (FIFO policy)
        self.turn_on_signals = 0

    # ------------------------------------------------------------ helpers
    def queued(self) -> int:
        return sum(len(q) for q in self.q_act)

    def _turn_on_check(self, k):
        if not self.active[k] or self.sender_on[k]:
            return
        if self.omega is None or self.queued() < self.omega:
            self.sender_on[k] = True
            self.turn_on_signals += 1

    # ------------------------------------------------------------ Alg. 2
    def put_act(self, k: int):
        """Returns (admitted, seq, slot)."""
        if not self.sender_on[k]:
            self.refused += 1
            return False, -1, -1
        slot = -1
        if self.free is not None:
            slot = self.free.pop()
        s = self.seq[k]
        self.seq[k] += 1
        self.q_act[k].append((s, slot, self.admissions))
        self.admissions += 1
        self.sender_on[k] = False
        self._turn_on_check(k)
        self.peak_queued = max(self.peak_queued, self.queued())
        return True, s, slot

    def put_model(self, k: int, t_k: int):
        self.q_model.append((k, t_k))

    # ------------------------------------------------------------ Alg. 3
    def get(self):
        """('model', k, t_k) | ('act', k, seq, slot) | None when nothing is queued."""
        if self.q_model:
            k, t_k = self.q_model.popleft()
            return ("model", k, t_k)
        best = None
        for k in range(self.K):
            if not self.q_act[k]:
                continue
            if best is None:
                best = k
            elif self.policy == "counter" and self.c[k] < self.c[best]:
                best = k
            elif self.policy == "fifo" and self.q_act[k][0][2] < self.q_act[best][0][2]:
                best = k
        if best is None:
            return None
        s, slot, _ = self.q_act[best].popleft()
        self.c[best] += 1
        self._turn_on_check(best)
        self.in_service = slot
        return ("act", best, s, slot)

    def release(self):
        """The batch in service has been trained on; its slot is free again."""
        if self.free is not None and self.in_service is not None and self.in_service >= 0:
            self.free.append(self.in_service)
        self.in_service = None

    # ------------------------------------------------------------ Alg. 4 versions
    def aggregate_version(self, t_k: int, max_delay=None):
        """Returns (applied, staleness).  t advances only when applied."""
        s = self.t - t_k
        if max_delay is not None and s > max_delay:
            return False, s
        self.t += 1
        return True, s

    # ------------------------------------------------------------ joining devices
    def add_device(self) -> int:
        """A device joining mid-run starts with c_k = 0 and its Sender on; the
        soft cap shrinks by one so the pool still holds every in-flight batch."""
        self.K += 1
        if self.n_slots is not None:
            self.omega = self.n_slots - self.K
            if self.omega < 1:
                raise ValueError("pool too small for the number of devices")
        self.q_act.append(deque())
        self.c.append(0)
        self.sender_on.append(True)
        self.seq.append(0)
        self.active.append(True)
        return self.K - 1

    def set_active(self, k: int, active: bool):
        """Device k leaves (active False: its Sender goes off and stays off) or
        rejoins (active True: its Sender starts on)."""
        self.active[k] = bool(active)
        self.sender_on[k] = bool(active)
