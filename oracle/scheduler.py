"""Oracle of the load-aware scheduler and its cost model (Sec. 3.2), in plain
Python. TEST INFRASTRUCTURE ONLY: used by ``tests/`` to check the library's
scheduler decision by decision; the library never loads it.

It takes the paper's steps in the paper's order, with these readings where
the text is silent:

* Cost model: linear interpolation of profiled points; on a 2-D grid of
  (requests, total context tokens) that is interpolation along the context
  axis at the two neighbouring request counts, then along the request axis.
  Outside the profiled range the nearest segment's line continues; an axis of
  one point is constant; a sub-batch with no request costs 0.
* Iteration time: T = L (max(T_l0, T_ca1) + max(T_l1 + T_ga0, T_ca0)) for two
  sub-batches, L (T_l0 + T_ga0) GPU-only; T_l of a sub-batch is taken at its
  token count (prefill tokens plus one per decoding request); T_ga / T_ca at
  the number of decoding requests and the sum of their context lengths
  including the new token.
* Memory: a request holds ceil(context / block_size) blocks; a decode needs
  room for one more token. Step 2 swaps out the most recently admitted GPU
  request first; if the CPU cache cannot take it the request is preempted and
  later prefilled again over its whole context. Swap-ins take the oldest CPU
  request first, stop at the first that does not fit with
  swap_in_reserve_blocks left free (no reserve while the GPU runs nothing),
  and do not happen in an iteration that swapped out.
* Activations: both sub-batches' linear-stage tokens together stay within
  max_batch_tokens (each sub-batch gets about half of a GPU-only batch); a
  single prefill longer than that still runs alone.
* Step 4 tries batch-1 before batch-0 (batch-1 holds most CPU decodes).
* Step 5 applies only when batch-1 has CPU decodes (with no CPU work the
  removal would stall admission and keep no CPU busy); it scans the prefills
  whose KV would be swapped out from the latest.
* Step 6 keeps the schedule with more requests per second, compared as
  x_two * T_gpu > x_gpu * T_two; ties keep the GPU-only schedule.
* If nothing at all would run while requests wait on the CPU, they run on the
  CPU without the balance constraints (progress).
"""
from __future__ import annotations

from collections import deque
from math import ceil


def _segment(axis, x):
    """Index i of the segment [axis[i], axis[i+1]] for x (nearest at the ends);
    None for a one-point axis."""
    if len(axis) < 2:
        return None
    i = 0
    while i + 1 < len(axis) and axis[i + 1] <= x:
        i += 1
    return min(i, len(axis) - 2)


def interp_curve(xs, ts, x):
    i = _segment(xs, x)
    if i is None:
        return ts[0]
    w = (x - xs[i]) / (xs[i + 1] - xs[i])
    return ts[i] + w * (ts[i + 1] - ts[i])


def interp_grid(bs, ss, table, b, s):
    i = _segment(bs, b)
    j = _segment(ss, s)
    ib = [0, 0] if i is None else [i, i + 1]
    js = [0, 0] if j is None else [j, j + 1]
    wb = 0.0 if i is None else (b - bs[i]) / (bs[i + 1] - bs[i])
    ws = 0.0 if j is None else (s - ss[j]) / (ss[j + 1] - ss[j])
    at_lo = table[ib[0]][js[0]] + ws * (table[ib[0]][js[1]] - table[ib[0]][js[0]])
    at_hi = table[ib[1]][js[0]] + ws * (table[ib[1]][js[1]] - table[ib[1]][js[0]])
    return at_lo + wb * (at_hi - at_lo)


class Request:
    def __init__(self, rid, prompt, output, arrival):
        self.rid, self.prompt, self.output, self.arrival = rid, prompt, output, arrival
        self.context = 0        # tokens with cached KV
        self.generated = 0      # output tokens so far
        self.todo_prefill = prompt
        self.state = "future"   # future / waiting / gpu / cpu / done


class OracleScheduler:
    def __init__(self, *, num_layers, block_size, gpu_blocks, cpu_blocks, max_batch_tokens,
                 t_ga, t_ca, t_l, swap_in_reserve_blocks=0, policy="neo"):
        self.L = num_layers
        self.bs = block_size
        self.gpu_cap = gpu_blocks
        self.cpu_cap = cpu_blocks
        self.act_cap = max_batch_tokens
        self.reserve = swap_in_reserve_blocks
        self.t_ga, self.t_ca, self.t_l = t_ga, t_ca, t_l  # (axes..., table)
        self.policy = policy
        self.pending = []
        self.waiting = deque()
        self.on_gpu = []
        self.on_cpu = []
        self.cpu_used = 0
        self.clock = 0.0
        self.total_tokens = 0

    # -- cost model
    def T_l(self, tokens):
        return 0.0 if tokens <= 0 else interp_curve(self.t_l[0], self.t_l[1], tokens)

    def T_ga(self, n, s):
        return 0.0 if n <= 0 else interp_grid(*self.t_ga, n, s)

    def T_ca(self, n, s):
        return 0.0 if n <= 0 else interp_grid(*self.t_ca, n, s)

    def nblocks(self, tokens):
        return ceil(tokens / self.bs)

    def add(self, rid, prompt, output, arrival=0.0):
        self.pending.append(Request(rid, prompt, output, max(arrival, self.clock)))

    def _arrive(self):
        self.pending.sort(key=lambda r: (r.arrival, r.rid))
        while self.pending and self.pending[0].arrival <= self.clock:
            r = self.pending.pop(0)
            r.state = "waiting"
            r.todo_prefill = r.prompt
            self.waiting.append(r)

    def step(self):
        self._arrive()
        if not self.waiting and not self.on_gpu and not self.on_cpu:
            if not self.pending:
                return None
            self.clock = max(self.clock, min(r.arrival for r in self.pending))
            self._arrive()

        # 1. Initialization: two empty batches.
        prefills, prefill_to_cpu = [], []
        gpu_decodes, cpu_b0, cpu_b1 = [], [], []
        swapped_out, swapped_in = [], []

        # 2. GPU decoding requests into batch-0; swap out until the GPU cache
        #    holds all new KV; swap in when there is ample space.
        need = sum(self.nblocks(r.context + 1) for r in self.on_gpu)
        while need > self.gpu_cap and self.on_gpu:
            r = self.on_gpu.pop()
            need -= self.nblocks(r.context + 1)
            if self.cpu_used + self.nblocks(r.context) <= self.cpu_cap:
                r.state = "cpu"
                self.cpu_used += self.nblocks(r.context)
                self.on_cpu.append(r)
                swapped_out.append(r)
            else:
                r.state = "waiting"
                r.todo_prefill = r.context
                r.context = 0
                self.waiting.appendleft(r)
        gpu_decodes = list(self.on_gpu)
        if not swapped_out:
            while self.on_cpu:
                r = self.on_cpu[0]
                keep_free = self.reserve if self.on_gpu else 0
                if need + self.nblocks(r.context + 1) + keep_free > self.gpu_cap:
                    break
                need += self.nblocks(r.context + 1)
                self.cpu_used -= self.nblocks(r.context)
                self.on_cpu.pop(0)
                r.state = "gpu"
                self.on_gpu.append(r)
                gpu_decodes.append(r)
                swapped_in.append(r)

        # 3. Prefills into batch-0 until the GPU cannot hold the activations;
        #    KV kept on the GPU if it fits, else swapped out to the CPU cache.
        tokens0 = len(gpu_decodes)
        cpu_after = self.cpu_used
        while self.waiting:
            r = self.waiting[0]
            if tokens0 > 0 and tokens0 + r.todo_prefill > self.act_cap:
                break
            nb = self.nblocks(r.todo_prefill)
            if need + nb <= self.gpu_cap:
                need += nb
                to_cpu = False
            elif cpu_after + nb <= self.cpu_cap:
                cpu_after += nb
                to_cpu = True
            else:
                break
            self.waiting.popleft()
            prefills.append(r)
            prefill_to_cpu.append(to_cpu)
            tokens0 += r.todo_prefill

        # 4. CPU decoding requests into batch-1 or batch-0 under
        #    T_ca1 <= T_l0 and T_ca0 <= T_l1 + T_ga0.
        ga0 = self.T_ga(len(gpu_decodes), sum(r.context + 1 for r in gpu_decodes))
        l0 = self.T_l(tokens0)
        l1 = ca0 = ca1 = 0.0
        ctx0 = ctx1 = 0
        if self.policy == "neo":
            for r in list(self.on_cpu):
                extra = self.nblocks(r.context + 1) - self.nblocks(r.context)
                if cpu_after + extra > self.cpu_cap:
                    continue
                if tokens0 + len(cpu_b1) + 1 > self.act_cap:
                    break
                new_ca1 = self.T_ca(len(cpu_b1) + 1, ctx1 + r.context + 1)
                new_l1 = self.T_l(len(cpu_b1) + 1)
                if new_ca1 <= l0 and ca0 <= new_l1 + ga0:
                    cpu_b1.append(r)
                    ctx1 += r.context + 1
                    ca1, l1 = new_ca1, new_l1
                    cpu_after += extra
                    continue
                new_ca0 = self.T_ca(len(cpu_b0) + 1, ctx0 + r.context + 1)
                new_l0 = self.T_l(tokens0 + 1)
                if new_ca0 <= l1 + ga0 and ca1 <= new_l0:
                    cpu_b0.append(r)
                    ctx0 += r.context + 1
                    ca0, l0 = new_ca0, new_l0
                    tokens0 += 1
                    cpu_after += extra

            # 5. Reduce prefilling requests that would swap out their KV.
            if cpu_b1:
                k = len(prefills) - 1
                while k >= 0:
                    if prefill_to_cpu[k]:
                        r = prefills[k]
                        smaller_l0 = self.T_l(tokens0 - r.todo_prefill)
                        if ca1 <= smaller_l0 and ca0 <= l1 + ga0:
                            tokens0 -= r.todo_prefill
                            l0 = smaller_l0
                            cpu_after -= self.nblocks(r.todo_prefill)
                            self.waiting.appendleft(r)
                            del prefills[k]
                            del prefill_to_cpu[k]
                    k -= 1

        if (self.policy == "neo" and not prefills and not gpu_decodes and not cpu_b0
                and not cpu_b1):
            for r in self.on_cpu:
                extra = self.nblocks(r.context + 1) - self.nblocks(r.context)
                if cpu_after + extra > self.cpu_cap:
                    continue
                if len(cpu_b1) + 1 > self.act_cap:
                    break
                cpu_b1.append(r)
                ctx1 += r.context + 1
                cpu_after += extra
            ca1 = self.T_ca(len(cpu_b1), ctx1)
            l1 = self.T_l(len(cpu_b1))
        if not prefills and not gpu_decodes and not cpu_b0 and not cpu_b1:
            raise RuntimeError("nothing can be scheduled")

        # 6. Decide: two-batch schedule vs GPU-only (batch-0 minus its CPU decodes).
        T_two = self.L * (max(l0, ca1) + max(l1 + ga0, ca0))
        T_gpu = self.L * (self.T_l(tokens0 - len(cpu_b0)) + ga0)
        x_two = len(prefills) + len(gpu_decodes) + len(cpu_b0) + len(cpu_b1)
        x_gpu = len(prefills) + len(gpu_decodes)
        if not cpu_b0 and not cpu_b1:
            two = False
        elif x_gpu == 0:
            two = True
        else:
            two = float(x_two) * T_gpu > float(x_gpu) * T_two
        T = T_two if two else T_gpu

        decision = {
            "mode": "two_batch" if two else "gpu_only",
            "prefill": [r.rid for r in prefills],
            "gpu_decode": [r.rid for r in gpu_decodes],
            "cpu_decode0": [r.rid for r in cpu_b0] if two else [],
            "cpu_decode1": [r.rid for r in cpu_b1] if two else [],
            "swap_out": [r.rid for r in swapped_out],
            "swap_in": [r.rid for r in swapped_in],
            "n_prefill_to_cpu": sum(prefill_to_cpu),
            "t_iter": T, "t_two_batch": T_two, "t_gpu_only": T_gpu,
            "t_l0": l0, "t_l1": l1, "t_ga0": ga0, "t_ca0": ca0, "t_ca1": ca1,
        }

        # Advance one token for everything that ran.
        for r, to_cpu in zip(prefills, prefill_to_cpu):
            r.context = r.todo_prefill
            r.generated += 1
            if r.generated >= r.output:
                r.state = "done"
                if to_cpu:
                    cpu_after -= self.nblocks(r.context)
            elif to_cpu:
                r.state = "cpu"
                self.on_cpu.append(r)
            else:
                r.state = "gpu"
                self.on_gpu.append(r)
        ran = gpu_decodes + ((cpu_b0 + cpu_b1) if two else [])
        for r in ran:
            r.context += 1
            r.generated += 1
            if r.generated >= r.output:
                if r.state == "cpu":
                    cpu_after -= self.nblocks(r.context)
                r.state = "done"
        if not two:
            for r in cpu_b0 + cpu_b1:
                cpu_after -= self.nblocks(r.context + 1) - self.nblocks(r.context)
        self.on_gpu = [r for r in self.on_gpu if r.state != "done"]
        self.on_cpu = [r for r in self.on_cpu if r.state != "done"]
        self.cpu_used = cpu_after
        self.clock += T
        x = x_two if two else x_gpu
        self.total_tokens += x
        decision["n_tokens"] = x
        decision["now"] = self.clock
        return decision
