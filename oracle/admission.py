"""Per-stage KV reservation and admission by observed lengths: plain model.

TEST INFRASTRUCTURE ONLY: never imported by the product path.

What the paper fixes. Each stage pool of the prefill / think / answer
pipeline reserves its own KV "chunk size" per request, in tokens (CS_T for
think, CS_A for answer; §IV-A, and the design-space table of §III-B lists 512 /
1024 / 2048). PSRoute sets CS_i to a rolling average of the token lengths
observed in that stage, instead of predicting each request's length; shorter
observed outputs shrink CS_i and admit more requests, longer ones admit fewer,
which keeps the KV cache from thrashing (§IV-D "PSRoute: adaptive admission
instead of prediction"). Memory-limited capacity is how many requests fit in
the KV cache at the current chunk size (§IV-C "System model").

Readings where the paper is silent (also listed in the design notes):
  * CS_i = mean of the last `window` completed requests' stage lengths,
    rounded up to a whole page (16 tokens) and clamped to [cs_min, cs_max];
    cs_initial before the first completion;
  * a request is admitted iff a sequence slot is free and the free pages
    cover its current context plus one chunk (ctx + CS_i tokens); waiting
    requests are taken in arrival order and admission stops at the first
    that does not fit;
  * a running sequence that outgrows its reservation reserves further whole
    chunks of the current CS_i; when the pool cannot cover that, the most
    recently admitted running sequence is preempted (its pages freed, the
    request goes back to the head of the waiting queue); a sequence that is
    itself the most recent one is preempted itself. That is the thrashing
    the adaptive chunk size is meant to avoid, counted as preemptions;
  * sequence ids are the lowest free slot, as the KV pool hands them out.

Every quantity is an integer: the model and the native scheduler must take
identical decisions on the same trace.
"""
PAGE = 16


def _pages(tokens: int) -> int:
    return (tokens + PAGE - 1) // PAGE


class AdmissionModel:
    def __init__(self, n_pages: int, max_seqs: int, max_pages_per_seq: int, window: int, cs_initial: int,
                 cs_min: int, cs_max: int):
        self.free = n_pages
        self.max_seqs = max_seqs
        self.max_pages = max_pages_per_seq
        self.window, self.cs_initial, self.cs_min, self.cs_max = window, cs_initial, cs_min, cs_max
        self.pages = {}      # seq -> reserved pages
        self.length = {}     # seq -> committed tokens
        self.order = {}      # seq -> admission counter
        self.counter = 0
        self.observed = []   # stage lengths of completed requests, oldest first

    # -------------------------------------------------------------- CS_i
    def chunk_size(self) -> int:
        if not self.observed:
            cs = self.cs_initial
        else:
            recent = self.observed[-self.window:]
            n, total = len(recent), sum(recent)
            cs = PAGE * ((total + PAGE * n - 1) // (PAGE * n))   # mean, rounded up to a page
        return min(max(cs, self.cs_min), self.cs_max)

    # -------------------------------------------------------------- admit
    def admit(self, ctx: int):
        """Sequence id if admitted (ctx + CS_i tokens reserved), else None."""
        want = _pages(ctx + self.chunk_size())
        if want > self.max_pages:
            raise ValueError("request larger than a sequence may ever hold")
        if want > self.free or len(self.pages) >= self.max_seqs:
            return None
        seq = min(s for s in range(self.max_seqs) if s not in self.pages)
        self.pages[seq], self.length[seq] = want, 0
        self.counter += 1
        self.order[seq] = self.counter
        self.free -= want
        return seq

    def commit(self, seq: int, n: int):
        assert self.length[seq] + n <= PAGE * self.pages[seq]
        self.length[seq] += n

    def _release(self, seq: int):
        self.free += self.pages.pop(seq)
        del self.length[seq], self.order[seq]

    # -------------------------------------------------------------- growth
    def reserve_step(self, seqs, n_tok):
        """Cover len + n for every listed sequence; returns preempted ids in
        preemption order."""
        preempted = []
        for s, n in zip(seqs, n_tok):
            if s not in self.pages:      # preempted earlier in this call
                continue
            need = self.length[s] + n
            cap = PAGE * self.pages[s]
            if need <= cap:
                continue
            cs = self.chunk_size()
            chunks = (need - cap + cs - 1) // cs
            want = _pages(cap + chunks * cs)
            if want > self.max_pages:
                want = self.max_pages
                if PAGE * want < need:
                    raise ValueError("sequence outgrows the longest a sequence may hold")
            extra = want - self.pages[s]
            while extra > self.free:
                victim = max(self.order, key=self.order.get)
                self._release(victim)
                preempted.append(victim)
                if victim == s:
                    break
            if s in self.pages:
                self.pages[s] = want
                self.free -= extra
        return preempted

    # -------------------------------------------------------------- finish
    def finish(self, seq: int, stage_tokens: int):
        self.observed.append(stage_tokens)
        self._release(seq)
