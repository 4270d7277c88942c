"""Plain reference of the task-aware KV block manager.

TEST INFRASTRUCTURE ONLY: the test suite is its only caller.  It shares no
code with the library's manager (paper_2504_03651_amd/csrc/kvm.cpp): blocks
are dicts, a full block is identified by the tuple of every token from the
start of its sequence through its end (no hashing), and every eviction scans
all evictable blocks for the minimum.

Rules, from Section 4.2 (KV cache manager design) and the KV cache manager
paragraph of Section 6:
  * a block referenced by a running task is never evicted (priority infinity);
  * an evictable block's priority is its reference count rc (registered
    offline prompts that contain its prefix, the running one included) when
    rc > 0, 1/2 when rc == 0 and its last task was online, 0 when rc == 0 and
    its last task was offline; the lowest priority is evicted first;
  * within a priority the least recently used block goes first (last access
    time).
Choices the paper leaves open, made the same way as the library documents
them: equal times evict the block deeper in its sequence first, then the lower
id; empty blocks (never filled, partial, or duplicates of a cached prefix) are
used before any eviction, lowest id first; a prompt whose every block is
cached still recomputes its last block; full blocks become visible to prefix
lookups at the end of the iteration that filled them (tick) or when their
sequence finishes; offline starts and appends may not raise the number of
held blocks above the offline limit.
"""
from __future__ import annotations

BS = 16
OK, E_INVALID, E_RANGE, E_NOSPACE = 0, -1, -2, -7
ONLINE, OFFLINE = 0, 1
EMPTY, HELD, CACHED = 0, 1, 2


class KVMOracle:
    def __init__(self, num_blocks: int, offline_limit: int | None = None):
        self.nb = num_blocks
        self.limit = num_blocks if offline_limit is None else offline_limit
        self.now = 0
        self.blocks = [self._fresh() for _ in range(num_blocks)]
        self.cache = {}      # prefix tuple -> block id (visible to lookups)
        self.rc = {}         # prefix tuple -> registered offline prompts
        self.reg = {}        # request -> list of prefix tuples
        self.seqs = {}       # sequence -> dict(task, tokens, blocks)
        self.pending = []    # blocks filled this iteration, in fill order
        self.copies = []
        self.evicted = []
        self.hits_tokens = 0
        self.n_evictions = 0

    @staticmethod
    def _fresh():
        return dict(state=EMPTY, holders=0, task=OFFLINE, lat=0, depth=0, prefix=None,
                    ntok=0, visible=False)

    # ------------------------------------------------------------ helpers
    def _rc(self, b):
        p = self.blocks[b]["prefix"]
        return self.rc.get(p, 0) if p is not None else 0

    def _priority2(self, b):
        r = self._rc(b)
        if r > 0:
            return 2 * r
        return 1 if self.blocks[b]["task"] == ONLINE else 0

    def _held(self):
        return sum(1 for x in self.blocks if x["state"] == HELD)

    def _available(self):
        return sum(1 for x in self.blocks if x["state"] != HELD)

    def _take(self):
        empties = [i for i, x in enumerate(self.blocks) if x["state"] == EMPTY]
        if empties:
            b = min(empties)
        else:
            cands = [i for i, x in enumerate(self.blocks) if x["state"] == CACHED]
            b = min(cands, key=lambda i: (self._priority2(i), self.blocks[i]["lat"],
                                          -self.blocks[i]["depth"], i))
            p = self.blocks[b]["prefix"]
            if self.cache.get(p) == b:
                del self.cache[p]
            self.evicted.append(b)
            self.n_evictions += 1
        self.blocks[b] = self._fresh()
        self.blocks[b].update(state=HELD, holders=1)
        return b

    def _stamp(self, b, task, depth):
        self.blocks[b].update(lat=self.now, task=task, depth=depth)

    def _publish(self, b):
        x = self.blocks[b]
        if x["prefix"] is None or x["visible"] or x["prefix"] in self.cache:
            return
        self.cache[x["prefix"]] = b
        x["visible"] = True

    # ------------------------------------------------------------ API
    def register_offline(self, req, tokens):
        if req in self.reg:
            return E_INVALID
        toks = tuple(int(t) for t in tokens)
        chain = [toks[:j + BS] for j in range(0, len(toks) - BS + 1, BS)]
        for p in chain:
            self.rc[p] = self.rc.get(p, 0) + 1
        self.reg[req] = chain
        return OK

    def unregister_offline(self, req):
        if req not in self.reg:
            return E_INVALID
        for p in self.reg.pop(req):
            self.rc[p] -= 1
            if self.rc[p] == 0:
                del self.rc[p]
        return OK

    def start(self, seq, task, tokens):
        toks = tuple(int(t) for t in tokens)
        n = len(toks)
        if n < 1 or task not in (ONLINE, OFFLINE) or seq in self.seqs:
            return E_INVALID, -1
        nfull, nblocks = n // BS, -(-n // BS)
        hits = []
        for j in range(nfull):
            b = self.cache.get(toks[:(j + 1) * BS])
            if b is None:
                break
            hits.append(b)
        if len(hits) == nfull and n % BS == 0 and hits:
            hits.pop()
        from_free = sum(1 for b in hits if self.blocks[b]["state"] == CACHED)
        n_new = nblocks - len(hits)
        if n_new > self._available() - from_free:
            return E_NOSPACE, -1
        if task == OFFLINE and self._held() + from_free + n_new > self.limit:
            return E_NOSPACE, -1
        blocks = []
        for j, b in enumerate(hits):
            x = self.blocks[b]
            x["state"] = HELD
            x["holders"] += 1
            self._stamp(b, task, j)
            blocks.append(b)
        for j in range(len(hits), nblocks):
            b = self._take()
            x = self.blocks[b]
            x["ntok"] = min(BS, n - j * BS)
            if j < nfull:
                x["prefix"] = toks[:(j + 1) * BS]
                self.pending.append(b)
            self._stamp(b, task, j)
            blocks.append(b)
        self.seqs[seq] = dict(task=task, tokens=list(toks), blocks=blocks)
        self.hits_tokens += BS * len(hits)
        return OK, BS * len(hits)

    def probe(self, tokens):
        toks = tuple(int(t) for t in tokens)
        n = len(toks)
        if n < 1:
            return E_INVALID, -1
        hits = 0
        for j in range(n // BS):
            if toks[:(j + 1) * BS] not in self.cache:
                break
            hits += 1
        if hits == n // BS and n % BS == 0 and hits:
            hits -= 1
        return OK, BS * hits

    def set_offline_limit(self, limit):
        if not 0 <= limit <= self.nb:
            return E_INVALID
        self.limit = limit
        return OK

    def append(self, seq, tokens):
        toks = [int(t) for t in tokens]
        if seq not in self.seqs or len(toks) < 1:
            return E_INVALID
        s = self.seqs[seq]
        ln = len(s["tokens"])
        cow = ln % BS != 0 and self.blocks[s["blocks"][-1]]["holders"] > 1
        n_new = -(-(ln + len(toks)) // BS) - len(s["blocks"]) + (1 if cow else 0)
        if n_new > self._available():
            return E_NOSPACE
        if s["task"] == OFFLINE and n_new > 0 and self._held() + n_new > self.limit:
            return E_NOSPACE
        if cow:
            src = s["blocks"][-1]
            dst = self._take()
            self.blocks[dst]["ntok"] = self.blocks[src]["ntok"]
            self.blocks[src]["holders"] -= 1
            s["blocks"][-1] = dst
            self.copies.append((src, dst))
        for t in toks:
            if len(s["tokens"]) % BS == 0:
                s["blocks"].append(self._take())
            s["tokens"].append(t)
            j = len(s["blocks"]) - 1
            b = s["blocks"][j]
            self.blocks[b]["ntok"] += 1
            self._stamp(b, s["task"], j)
            if self.blocks[b]["ntok"] == BS:
                self.blocks[b]["prefix"] = tuple(s["tokens"])
                self.pending.append(b)
        return OK

    def fork(self, parent, child):
        if parent not in self.seqs or child in self.seqs:
            return E_INVALID
        p = self.seqs[parent]
        c = dict(task=p["task"], tokens=list(p["tokens"]), blocks=list(p["blocks"]))
        for j, b in enumerate(c["blocks"]):
            self.blocks[b]["holders"] += 1
            self._stamp(b, c["task"], j)
        self.seqs[child] = c
        return OK

    def finish(self, seq):
        if seq not in self.seqs:
            return E_INVALID
        s = self.seqs.pop(seq)
        for b in s["blocks"]:
            self._publish(b)
        for j in range(len(s["blocks"]) - 1, -1, -1):
            b = s["blocks"][j]
            x = self.blocks[b]
            self._stamp(b, s["task"], j)
            x["holders"] -= 1
            if x["holders"] > 0:
                continue
            if x["visible"]:
                x["state"] = CACHED
            else:
                self.blocks[b] = self._fresh()
        return OK

    def tick(self):
        for b in self.pending:
            self._publish(b)
        self.pending = []
        self.now += 1
        return OK

    def block_tables(self, seqs, mbr):
        for q in seqs:
            if q not in self.seqs:
                return E_INVALID, None
            if len(self.seqs[q]["blocks"]) > mbr:
                return E_RANGE, None
        bt = [[-1] * mbr for _ in seqs]
        sl = []
        for r, q in enumerate(seqs):
            s = self.seqs[q]
            bt[r][:len(s["blocks"])] = s["blocks"]
            sl.append(len(s["tokens"]))
        return OK, (bt, sl)

    def take_copies(self):
        out, self.copies = self.copies, []
        return out

    def take_evictions(self):
        out, self.evicted = self.evicted, []
        return out

    def block_info(self, b):
        x = self.blocks[b]
        return dict(state=x["state"], holders=x["holders"], rc=self._rc(b), task=x["task"],
                    lat=x["lat"], priority2=self._priority2(b) if x["state"] == CACHED else -1,
                    depth=x["depth"])

    def stats(self):
        return dict(empty=sum(1 for x in self.blocks if x["state"] == EMPTY), held=self._held(),
                    cached=sum(1 for x in self.blocks if x["state"] == CACHED),
                    running=len(self.seqs), now=self.now, hits_tokens=self.hits_tokens,
                    evictions=self.n_evictions,
                    cached_reusable=sum(1 for b, x in enumerate(self.blocks)
                                        if x["state"] == CACHED and self._rc(b) > 0))
