"""Plain-Python model of the device batch insert (the round structure of the
merge kernels) on the flattened union layout.  Used by CPU tests to check the
algorithm against the oracle; it is not called by the library."""
from __future__ import annotations

import numpy as np


class FlatForest:
    def __init__(self, img, P):
        n = img["nodes"].shape[0]
        self.P = P
        self.nodes = []
        for i in range(n):
            r = img["nodes"][i]
            mask = 0
            for w, x in enumerate(img["masks"][i].tolist()):
                mask |= int(x) << (64 * w)
            self.nodes.append(dict(tok=int(r[0]), off=int(np.uint32(r[1])), len=int(r[2]), cb=int(r[3]),
                                   cc=int(r[4]), aux=0, mask=mask))
        self.pool = img["pool"].tolist()
        self.moved = {}
        self.stamp = 0

    # -- the walk of merge_walk_kernel
    def find_child(self, x, t):
        nx = self.nodes[x]
        for j in range(nx["cc"]):
            if self.nodes[nx["cb"] + j]["tok"] == t:
                return nx["cb"] + j
        return -1

    def walk(self, s, p):
        """Classify an insert; on the way, set its peer bit in every node it
        passes through whole (the root included)."""
        x, d = 0, 0
        self.nodes[0]["mask"] |= 1 << p
        while True:
            if d == len(s):
                return ("done", x, -1, 0, d, 0)
            t = s[d]
            c = self.find_child(x, t)
            if c < 0:
                return ("add", x, -1, 0, d, t)
            nc = self.nodes[c]
            n = min(nc["len"], len(s) - d)
            l = 0
            while l < n and self.pool[nc["off"] + l] == s[d + l]:
                l += 1
            if l == nc["len"]:
                x, d = c, d + l
                nc["mask"] |= 1 << p
                continue
            return ("split", x, c, l, d, t)

    def alloc_pool(self, toks):
        off = len(self.pool)
        self.pool.extend(int(t) for t in toks)
        return off

    def merge(self, seqs, peers):
        """Rounds as the device runs them: walk every unfinished insert; then,
        from that one walk, the add phase (the first insert of each
        (parent, token) slot adds a leaf to its parent's rebuilt block) and
        the split phase (the lowest insert per edge cuts it; the edge's record
        is found through its move stamp if the add phase moved it).  Winners
        are done; everyone else walks again.  Peer bits: each walk sets them on
        its path, a new leaf holds its winner's, a cut edge's upper part adds
        the winner's, and records keep theirs when they move or split."""
        n = len(seqs)
        st = [None] * n
        active = [True] * n
        while True:
            for i in range(n):
                if active[i]:
                    st[i] = self.walk(seqs[i], peers[i])
                    if st[i][0] == "done":
                        active[i] = False
            splits = [i for i in range(n) if active[i] and st[i][0] == "split"]
            adds = [i for i in range(n) if active[i] and st[i][0] == "add"]
            if not splits and not adds:
                break
            stamp = 0
            if adds:
                self.stamp += 1
                stamp = self.stamp
                order = sorted(adds, key=lambda i: (st[i][1], st[i][5], i))
                groups = {}
                for i in order:
                    groups.setdefault(st[i][1], []).append(i)
                new_blocks = {}
                for x, members in groups.items():  # build (reads old records only)
                    winners, seen = [], set()
                    for i in members:
                        if st[i][5] not in seen:
                            seen.add(st[i][5])
                            winners.append(i)
                    nx = self.nodes[x]
                    old = [dict(self.nodes[nx["cb"] + j]) for j in range(nx["cc"])]
                    leaves = []
                    for i in winners:
                        s, d = seqs[i], st[i][4]
                        leaves.append(dict(tok=int(s[d]), off=self.alloc_pool(s[d:]), len=len(s) - d, cb=0, cc=0,
                                           aux=0, mask=1 << peers[i]))
                        active[i] = False
                    block = sorted(old + leaves, key=lambda r: r["tok"])
                    nb = len(self.nodes)
                    self.nodes.extend(block)
                    for j in range(nx["cc"]):
                        src = nx["cb"] + j
                        pos = nb + [k for k, r in enumerate(block) if r["tok"] == self.nodes[src]["tok"]][0]
                        self.moved[src] = (self.stamp, pos)
                    new_blocks[x] = (nb, len(block))
                for x, (nb, cnt) in new_blocks.items():  # fix
                    stp, pos = self.moved.get(x, (0, x))
                    pos = pos if stp == self.stamp else x
                    self.nodes[pos]["cb"], self.nodes[pos]["cc"] = nb, cnt

            def where(c):
                stp, pos = self.moved.get(c, (0, c))
                return pos if stamp and stp == stamp else c

            if splits:
                for i in splits:  # claim: lowest index per edge
                    c = where(st[i][2])
                    self.nodes[c]["aux"] = max(self.nodes[c]["aux"], 2 ** 31 - 1 - i)
                for i in splits:
                    _, x, c, l, d, t = st[i]
                    c = where(c)
                    if self.nodes[c]["aux"] != 2 ** 31 - 1 - i:
                        continue
                    s = seqs[i]
                    rest = len(s) - d - l
                    old = dict(self.nodes[c])
                    lower = dict(old, off=old["off"] + l, len=old["len"] - l, aux=0)
                    lower["tok"] = self.pool[lower["off"]]
                    nb = len(self.nodes)
                    block = [lower]
                    if rest > 0:
                        leaf = dict(tok=int(s[d + l]), off=self.alloc_pool(s[d + l:]), len=rest, cb=0, cc=0,
                                    aux=0, mask=1 << peers[i])
                        block = sorted([lower, leaf], key=lambda r: r["tok"])
                    self.nodes.extend(block)
                    self.nodes[c] = dict(old, len=l, cb=nb, cc=len(block), aux=0, mask=old["mask"] | (1 << peers[i]))
                    active[i] = False
        for i in range(n):  # every sequence ends at a node holding its peer
            s, p = seqs[i], peers[i]
            x, d = 0, 0
            while d < len(s):
                c = self.find_child(x, s[d])
                assert c >= 0 and d + self.nodes[c]["len"] <= len(s), "sequence does not end at a node"
                x, d = c, d + self.nodes[c]["len"]
                assert (self.nodes[x]["mask"] >> p) & 1, "a node on the path lacks the peer's bit"

    def clear_peer(self, p):
        for r in self.nodes:
            r["mask"] &= ~(1 << p)

    def route(self, q):
        alive = (1 << self.P) - 1
        m = [0] * self.P
        x, d = 0, 0
        while d < len(q):
            c = self.find_child(x, q[d])
            if c < 0:
                break
            nm = alive & self.nodes[c]["mask"]
            for p in range(self.P):
                if (alive >> p) & 1 and not (nm >> p) & 1:
                    m[p] = d
            alive = nm
            if not alive:
                break
            nc = self.nodes[c]
            l = 0
            while l < nc["len"] and d + l < len(q) and self.pool[nc["off"] + l] == q[d + l]:
                l += 1
            d += l
            if l < nc["len"]:
                break
            x = c
        for p in range(self.P):
            if (alive >> p) & 1:
                m[p] = d
        return m
