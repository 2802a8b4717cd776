"""Host simulator of conversation-level disaggregated serving over this library's kernels.

It replays an agentic trace through the placement rules of the library -- every turn-1 prefill is
admitted on the prefiller's expected backlog (``cs_sched_admit``) and, after it, the conversation
is bound once to the decoder with the lowest KV occupancy that can hold it
(``cs_place_least_occupied``) -- and times the GPU work with a cost model of the kernels as
measured on one MI355X. No kernel runs; it shows how the paper's two phases look on this hardware
(Section 3.1: turn-1 prefill is compute-bound and quadratic in the input length, later turns
reuse the cached prefix; Section 3.2 and its collocation experiment: the decode side is
memory-bound and, with enough active KV, sets the iteration time; Section 4.2: reactive placement
on the prefill curve and the decoders' occupancy).

Model
-----
* One prefiller GPU runs the admitted turn-1 prefills one after another; a prefill of L tokens
  takes the measured curve t(L) (all layers). A conversation whose expected wait exceeds
  ``max_wait_s`` is refused -- the paper routes it elsewhere; here it retries, in arrival order,
  whenever a prefill completes. Its turn-1 TTFT is its prefill's end minus its arrival (the first
  token comes out of the prefill).
* After the prefill the conversation is bound to a decoder (least occupied with room for its
  pages); if none has room it waits until pages are freed. The KV moves once: pack, one link
  between the GPUs, unpack.
* Each decoder runs iterations back to back while it has work. An iteration takes the pending
  extend chunks in arrival order (at most ``extend_budget`` tokens, the first always) and one
  decode token of every conversation in its decode phase; it lasts the decode time of the
  iteration's active KV plus the extend time of its chunks. A later turn's TTFT is the end of the
  iteration that ran its extend chunk minus the arrival of its appended tokens. A conversation
  whose turn's decodes are done is idle for ``tool_s`` (the agent's tool call) and keeps its pages;
  after its last turn it ends and its pages return.
* When an iteration's page growth does not fit, extend chunks are held back first; if the decode
  tokens alone do not fit, the most recently bound conversation is swapped out to host memory
  (pack over ``host_gbs``) and swapped back into the same decoder once it has room again (the
  paper is silent on this; a serving engine preempts this way).

The cost model's defaults are this library's kernels measured on one MI355X (32 layers of a
Llama-3-8B-shaped model: 32 query / 8 KV heads, head_dim 128): the turn-1 prefill curve per layer,
the decode step's fixed cost per layer and its marginal bandwidth, the extend rate, pack/unpack.
``CostModel.from_bench`` takes them from a bench.py JSON line instead.
"""
from __future__ import annotations

import heapq
import math
from dataclasses import dataclass, field

from .conserve import PAGE_TOKENS, Scheduler, place_least_occupied


def pages_for(tokens: int) -> int:
    return -(-int(tokens) // PAGE_TOKENS)


@dataclass(frozen=True)
class CostModel:
    """Seconds of GPU work of the hot path, all layers. Rates: GB/s, TFLOP/s; inf makes a term 0."""
    n_layers: int = 32
    n_q_heads: int = 32
    n_kv_heads: int = 8
    head_dim: int = 128
    prefill_curve: tuple = (1.57e-5, 4.94e-9, 6.81e-12)  # one layer: c0 + c1 L + c2 L^2 seconds
    decode_fixed_s: float = 2.0e-5     # per layer and iteration
    decode_gbs: float = 6810.0         # marginal KV read rate of the decode step
    extend_fixed_s: float = 2.0e-5     # per layer and iteration with extend work
    extend_tflops: float = 1200.0
    move_gbs: float = 5000.0           # pack / unpack, read + write bytes
    link_gbs: float = 153.0            # one xGMI link, prefiller -> decoder
    host_gbs: float = 50.0             # device <-> host, for swapping a conversation out and in

    @property
    def kv_bytes_token(self) -> int:
        """K and V of one token, all layers (bf16)."""
        return self.n_layers * 2 * self.n_kv_heads * self.head_dim * 2

    def prefill_s(self, L: int) -> float:
        c0, c1, c2 = self.prefill_curve
        return self.n_layers * (c0 + L * (c1 + L * c2))

    def transfer_s(self, L: int) -> float:
        b = L * self.kv_bytes_token
        return 2 * (2 * b) / (self.move_gbs * 1e9) + b / (self.link_gbs * 1e9)

    def swap_s(self, L: int) -> float:
        b = L * self.kv_bytes_token
        return 2 * b / (self.move_gbs * 1e9) + b / (self.host_gbs * 1e9)

    def decode_s(self, active_tokens: int, n_convs: int) -> float:
        if n_convs == 0:
            return 0.0
        per_layer = active_tokens * self.kv_bytes_token / self.n_layers
        return self.n_layers * (self.decode_fixed_s + per_layer / (self.decode_gbs * 1e9))

    def extend_s(self, chunks) -> float:
        """chunks: [(prefix P, new tokens n)]; work = 4 d Hq (n P + n (n + 1) / 2) FLOP per layer."""
        if not chunks:
            return 0.0
        pairs = sum(n * P + n * (n + 1) // 2 for P, n in chunks)
        flops = 4 * self.head_dim * self.n_q_heads * pairs
        return self.n_layers * (self.extend_fixed_s + flops / (self.extend_tflops * 1e12))

    @classmethod
    def from_bench(cls, line: dict, **kw) -> "CostModel":
        """Rates from a bench.py JSON line (its components prefill_curve, decode_curve, extend,
        pack and unpack), which measure one layer of the same attention shape."""
        c = line.get("components", line)
        args = dict(kw)
        if "prefill_curve" in c:
            args["prefill_curve"] = tuple(c["prefill_curve"]["coef_s"])
        if "decode_curve" in c:
            args["decode_fixed_s"] = c["decode_curve"]["fixed_ms"] * 1e-3
            args["decode_gbs"] = c["decode_curve"]["marginal_gbs"]
        if "extend" in c:
            args["extend_tflops"] = c["extend"]["roofline"]["achieved"]
        if "pack" in c and "unpack" in c:
            args["move_gbs"] = min(c["pack"]["gbs"], c["unpack"]["gbs"])
        return cls(**args)


@dataclass
class ConvSpec:
    """One conversation of the trace: turn-1 prompt, appended tokens of turns 2.., decoded tokens
    of every turn (len(decodes) = turns), arrival time in seconds."""
    turn1: int
    appends: list
    decodes: list
    arrival: float = 0.0


@dataclass
class _Conv:
    idx: int
    spec: ConvSpec
    length: int = 0
    pages: int = 0
    turn: int = 0
    left: int = 0
    phase: str = "arriving"    # arriving refused prefill bind transfer decode tool append swapped done
    decoder: int = -1
    bound_at: float = 0.0
    turn_start: float = 0.0
    ttft: list = field(default_factory=list)       # per turn
    context: list = field(default_factory=list)    # cached tokens before each later turn's append
    finish: float = math.nan
    swaps: int = 0


@dataclass
class Iteration:
    decoder: int
    start: float
    decode_s: float
    extend_s: float
    active_tokens: int       # KV tokens the decode part reads (every decoding conversation, +1)
    n_decode: int
    extend_tokens: int

    @property
    def duration(self) -> float:
        return self.decode_s + self.extend_s

    @property
    def decode_dominated(self) -> bool:
        return self.decode_s >= self.extend_s


class Simulator:
    """Discrete-event simulation; ``run()`` returns the summary dict (see ``summary``)."""

    def __init__(self, trace, cost: CostModel = CostModel(), n_decoders: int = 2,
                 pages_per_decoder: int = 100_000, max_wait_s: float = 60.0, tool_s: float = 0.0,
                 extend_budget: int = 8192):
        self.cost = cost
        self.convs = [_Conv(i, s) for i, s in enumerate(trace)]
        self.n_dec = n_decoders
        self.cap = [int(pages_per_decoder)] * n_decoders
        self.used = [0] * n_decoders
        self.tool_s = tool_s
        self.extend_budget = extend_budget
        # admission-only scheduler on the all-layer prefill curve; binding reads the simulated pages
        self.sched = Scheduler(tuple(cost.n_layers * c for c in cost.prefill_curve), max_wait_s)
        self.events = []
        self._seq = 0
        self.refused = []            # FIFO of conversations refused admission
        self.bind_wait = []          # FIFO of prefilled conversations no decoder can hold yet
        self.live = [[] for _ in range(n_decoders)]
        self.busy = [False] * n_decoders
        self.swapped = [[] for _ in range(n_decoders)]
        self.copy_s = [0.0] * n_decoders    # swap copies to charge to a decoder's next iteration
        self.iterations = []
        self.refusals = 0
        self.now = 0.0

    # -- event plumbing ---------------------------------------------------------------------------
    def _push(self, t, kind, *data):
        heapq.heappush(self.events, (t, self._seq, kind, data))
        self._seq += 1

    def run(self) -> dict:
        for c in self.convs:
            self._push(c.spec.arrival, "arrive", c)
        while self.events:
            t, _, kind, data = heapq.heappop(self.events)
            self.now = t
            getattr(self, "_on_" + kind)(*data)
        self.sched.close()
        return self.summary()

    # -- prefiller --------------------------------------------------------------------------------
    def _admit(self, c) -> bool:
        got = self.sched.admit(c.spec.turn1, self.now)
        if got is None:
            return False
        c.phase = "prefill"
        self._push(got[1], "prefill_done", c)
        return True

    def _on_arrive(self, c):
        if self.refused or not self._admit(c):
            c.phase = "refused"
            self.refused.append(c)
            self.refusals += 1

    def _on_prefill_done(self, c):
        c.length = c.spec.turn1
        c.ttft.append(self.now - c.spec.arrival)
        c.phase = "bind"
        self.bind_wait.append(c)
        self._bind_waiting()
        while self.refused and self._admit(self.refused[0]):
            self.refused.pop(0)

    # -- binding and transfer ---------------------------------------------------------------------
    def _bind_waiting(self):
        while self.bind_wait:
            c = self.bind_wait[0]
            need = pages_for(c.length)
            free = [self.cap[i] - self.used[i] for i in range(self.n_dec)]
            d = place_least_occupied(self.used, free, need)
            if d < 0:
                return
            self.bind_wait.pop(0)
            c.decoder, c.pages, c.bound_at, c.phase = d, need, self.now, "transfer"
            self.used[d] += need
            self._push(self.now + self.cost.transfer_s(c.length), "transfer_done", c)

    def _on_transfer_done(self, c):
        c.phase, c.turn, c.left = "decode", 0, c.spec.decodes[0]
        self.live[c.decoder].append(c)
        self._kick(c.decoder)

    # -- decoders ---------------------------------------------------------------------------------
    def _kick(self, d):
        if not self.busy[d]:
            self._start_iteration(d)

    def _start_iteration(self, d):
        self._resume_swapped(d)
        live = self.live[d]
        ext = sorted((c for c in live if c.phase == "append"), key=lambda c: (c.turn_start, c.idx))
        chunks, tokens = [], 0
        for c in ext:
            n = c.spec.appends[c.turn - 1]
            if chunks and tokens + n > self.extend_budget:
                break
            chunks.append(c)
            tokens += n
        while True:
            dec = [c for c in live if c.phase == "decode"]
            grow = sum(pages_for(c.length + 1) - c.pages for c in dec)
            grow += sum(pages_for(c.length + c.spec.appends[c.turn - 1]) - c.pages for c in chunks)
            if grow <= self.cap[d] - self.used[d]:
                break
            if chunks:                       # hold extend chunks back first
                chunks.pop()
            elif dec:                        # then preempt the most recently bound conversation
                self._swap_out(d)
            else:
                break
        dec = [c for c in live if c.phase == "decode"]
        if not dec and not chunks:
            self.busy[d] = False
            return
        for c in dec + chunks:
            n = 1 if c.phase == "decode" else c.spec.appends[c.turn - 1]
            g = pages_for(c.length + n) - c.pages
            c.pages += g
            self.used[d] += g
        assert self.used[d] <= self.cap[d], "page accounting exceeded the decoder's capacity"
        it = Iteration(d, self.now,
                       self.cost.decode_s(sum(c.length + 1 for c in dec), len(dec)),
                       self.cost.extend_s([(c.length, c.spec.appends[c.turn - 1]) for c in chunks]),
                       sum(c.length + 1 for c in dec), len(dec),
                       sum(c.spec.appends[c.turn - 1] for c in chunks))
        self.iterations.append(it)
        self.busy[d] = True
        extra, self.copy_s[d] = self.copy_s[d], 0.0
        self._push(self.now + it.duration + extra, "iteration_done", d, dec, chunks)

    def _on_iteration_done(self, d, dec, chunks):
        for c in chunks:
            c.context.append(c.length)
            c.length += c.spec.appends[c.turn - 1]
            c.ttft.append(self.now - c.turn_start)
            c.phase, c.left = "decode", c.spec.decodes[c.turn]
        freed = False
        for c in dec:
            c.length += 1
            c.left -= 1
            if c.left > 0:
                continue
            c.turn += 1
            if c.turn == len(c.spec.decodes):
                c.phase, c.finish = "done", self.now
                self.live[d].remove(c)
                self.used[d] -= c.pages
                c.pages = 0
                freed = True
            else:
                c.phase = "tool"
                self._push(self.now + self.tool_s, "append_arrive", c)
        if freed:
            self._bind_waiting()
        self._start_iteration(d)

    def _on_append_arrive(self, c):
        c.phase, c.turn_start = "append", self.now
        self._kick(c.decoder)

    # -- preemption (swap to host and back) -------------------------------------------------------
    def _swap_out(self, d):
        c = max((x for x in self.live[d] if x.phase == "decode"), key=lambda x: (x.bound_at, x.idx))
        self.live[d].remove(c)
        self.used[d] -= c.pages
        c.pages = 0
        c.phase, c.swaps = "swapped", c.swaps + 1
        self.swapped[d].append(c)
        self.copy_s[d] += self.cost.swap_s(c.length)

    def _resume_swapped(self, d):
        """Swapped conversations come back, in the order they left, once their pages plus one
        page of growth for every live conversation fit; the copy-in is charged to the decoder."""
        while self.swapped[d]:
            c = self.swapped[d][0]
            need = pages_for(c.length)
            if self.cap[d] - self.used[d] < need + len(self.live[d]) + 1:
                return
            self.swapped[d].pop(0)
            c.pages, c.phase = need, "decode"
            self.used[d] += need
            self.live[d].append(c)
            self.copy_s[d] += self.cost.swap_s(c.length)

    # -- results ----------------------------------------------------------------------------------
    def decode_dominance(self, edges) -> list:
        """For iterations that ran extend work beside decoding, binned by active KV tokens at the
        bin edges given: (lo, hi, iterations, share whose decode part took at least as long as
        the extend part)."""
        out = []
        for lo, hi in zip(edges[:-1], edges[1:]):
            its = [i for i in self.iterations if i.extend_tokens and i.n_decode and lo <= i.active_tokens < hi]
            out.append((lo, hi, len(its), sum(i.decode_dominated for i in its) / len(its) if its else None))
        return out

    def summary(self) -> dict:
        done = [c for c in self.convs if c.phase == "done"]
        tokens = sum(c.spec.turn1 + sum(c.spec.appends) + sum(c.spec.decodes) for c in done)
        decoded = sum(sum(c.spec.decodes) for c in done)
        t0 = min((c.spec.arrival for c in self.convs), default=0.0)
        span = max((c.finish for c in done), default=t0) - t0
        return {"conversations": len(self.convs), "completed": len(done), "refusals": self.refusals,
                "swaps": sum(c.swaps for c in self.convs), "makespan_s": span,
                "tokens_per_s": tokens / span if span > 0 else None,
                "decode_tokens_per_s": decoded / span if span > 0 else None,
                "turn1_ttft": [(c.spec.turn1, c.ttft[0]) for c in done],
                "later_ttft": [(P, c.spec.appends[k], t) for c in done
                               for k, (P, t) in enumerate(zip(c.context, c.ttft[1:]))],
                "finish": [c.finish for c in self.convs],
                "iterations": len(self.iterations),
                "decoder_tokens": [sum(c.spec.turn1 + sum(c.spec.appends) + sum(c.spec.decodes)
                                       for c in done if c.decoder == d) for d in range(self.n_dec)]}
