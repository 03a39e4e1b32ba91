"""fp64 CPU oracle of the multi-commit lifecycle driver (Algorithm 1).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: only ``tests/``,
``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may import
it, and it shares no code with the HIP library.

``Agent`` keeps the state Algorithm 1 carries across the turns of one agent
episode and composes the per-commit steps of ``commitkv_oracle``:

* the resident cache: keys and values of every layer (bf16 bits, copied
  verbatim) and absolute positions, in ascending position order;
* the events seen so far (kind, first position, length);
* the pending commit: the pages measured before the last commit and their
  pre-commit effects R^-, until its post-commit window is measured;
* the retirement set D_c (Sec. 3.3), pages by absolute position.

Readings taken where the paper leaves the driver open (the library's driver
takes the same ones):

* L1  pages: every tool-call and observation event is cut into pages of at
      most G tokens from its first token (Sec. 3.1); a page is identified by
      its absolute positions, so it survives compaction.
* L2  E_c at a commit: the pages of the events seen so far whose tokens are
      all resident and that are not in D_c; with a scan cap m (Sec. 4.1:
      64), the m pages of largest start position.
* L3  the pre-commit window is the last W tokens of the tool call; the
      post-commit window is the first W tokens of the reasoning that follows
      the observation (Eq. (5)).  The post measurement covers the pages of
      the pending commit that are still fully resident, with percentiles
      among them; their R^- is the value stored at the commit.
* L4  pending pages are protected at every checkpoint until the post
      measurement; one that is no longer fully resident is not (its
      post-commit effect can no longer be measured).
* L5  a checkpoint follows every C decoded tokens (Sec. 4.1: 128).  Its base
      score is the token mass of the last W resident tokens as the window,
      on one designated scoring layer, pooled over pool_kernel tokens when
      that is above 1 (reading R12); one index set serves every layer
      (Eq. (4)).  With at most B resident tokens and no resident retired
      token a checkpoint changes nothing.
* L6  accepted pages join D_c (Algorithm 1) and stay resident until the next
      checkpoint removes their tokens; a page with no resident token left
      leaves D_c.
"""
from __future__ import annotations

import numpy as np

from . import commitkv_oracle as O

TOOL_CALL, OBSERVATION = 1, 2      # event kinds that are cut into pages (Sec. 3.1)


class Agent:
    def __init__(self, n_layers, n_kv_heads, head_dim, page_size, budget, eta=0.125,
                 max_pending_pages=16, max_scan_pages=64, keep_recent=0, score_layer=0,
                 thresholds=None, ablation=(), method="closed", pool_kernel=0, pool_mode="max"):
        self.G = page_size
        self.B = budget
        self.eta = eta
        self.max_pending = max_pending_pages
        self.max_scan = max_scan_pages
        self.keep_recent = keep_recent
        self.score_layer = score_layer
        self.th = dict(O.PAPER_THRESHOLDS if thresholds is None else thresholds)
        self.ablation = tuple(ablation)
        self.method = method
        self.pool = (pool_kernel, pool_mode)
        self.K = [np.zeros((n_kv_heads, 0, head_dim), np.uint16) for _ in range(n_layers)]
        self.V = [np.zeros((n_kv_heads, 0, head_dim), np.uint16) for _ in range(n_layers)]
        self.pos = np.zeros(0, np.int64)
        self.events = []          # [kind, start, length]
        self.pending = None       # (pages, r_pre)
        self.retired = []         # D_c
        self.decoded = 0

    # ------------------------------------------------------------ the cache
    def append(self, kind, p0, p1, k_layers, v_layers, decoded=False, begins_event=True):
        """Tokens at positions [p0, p1) enter the cache (k_layers[l]: [Hkv, n, d])."""
        if self.pos.size and p0 <= self.pos[-1]:
            raise ValueError("positions must increase")
        for l in range(len(self.K)):
            self.K[l] = np.concatenate([self.K[l], k_layers[l]], axis=1)
            self.V[l] = np.concatenate([self.V[l], v_layers[l]], axis=1)
        self.pos = np.concatenate([self.pos, np.arange(p0, p1)])
        if begins_event or not self.events or self.events[-1][0] != kind:
            self.events.append([kind, p0, p1 - p0])
        else:
            self.events[-1][2] = p1 - self.events[-1][1]
        if decoded:
            self.decoded += p1 - p0

    def span(self, page):
        """Resident index range [i0, i1) of the positions of ``page``."""
        s, ln = page
        i0 = int(np.searchsorted(self.pos, s, side="left"))
        i1 = int(np.searchsorted(self.pos, s + ln, side="left"))
        return i0, i1

    def fully_resident(self, page):
        i0, i1 = self.span(page)
        return i1 - i0 == page[1]

    def ranges(self, pages):
        return [(self.span(p)[0], p[1]) for p in pages]

    # ------------------------------------------------------------ pages
    def agent_pages(self):
        """L1: pages of every tool-call and observation event, by position."""
        out = []
        for kind, st, ln in self.events:
            if kind in (TOOL_CALL, OBSERVATION):
                out += [(st + off, min(self.G, ln - off)) for off in range(0, ln, self.G)]
        return out

    def eligible(self):
        """L2: E_c, fully resident and not retired, the most recent max_scan."""
        ret = set(self.retired)
        pages = [p for p in self.agent_pages() if p not in ret and self.fully_resident(p)]
        if self.max_scan and self.max_scan > 0:
            pages = pages[-self.max_scan:]
        return pages

    def _layer(self):
        l = self.score_layer
        return self.K[l], self.V[l], self.pos

    # ------------------------------------------------------------ Algorithm 1
    def commit(self, Q, qpos):
        """Pre-commit measurement over E_c (Eq. (5)-(8), window Q^-)."""
        pages = self.eligible()
        K, V, pos = self._layer()
        R_pre = O.page_effects(K, V, pos, Q, qpos, self.ranges(pages), method=self.method)[0] \
            if pages else np.zeros(0)
        self.pending = (pages, R_pre)
        return dict(pages=pages, R_pre=R_pre)

    def post_measure(self, Q, qpos):
        """L3: post-commit effects and classification of the pending pages
        that are still fully resident (Eq. (8)-(10))."""
        pages, r_pre = self.pending if self.pending else ([], np.zeros(0))
        keep = [j for j, p in enumerate(pages) if self.fully_resident(p)]
        pages = [pages[j] for j in keep]
        r_pre = np.asarray(r_pre)[keep]
        K, V, pos = self._layer()
        rng = self.ranges(pages)
        if pages:
            R_post = O.page_effects(K, V, pos, Q, qpos, rng, method=self.method)[0]
        else:
            R_post = np.zeros(0)
        th = {k: self.th[k] for k in ("tau_use", "tau_dead", "rho_use", "rho_dead")}
        lam, Pm, Pp, cand = O.classify(r_pre, R_post, [s for s, _ in rng], ablation=self.ablation, **th)
        return dict(pages=pages, R_pre=r_pre, R_post=R_post, lam=lam, P_pre=Pm, P_post=Pp,
                    cand=np.asarray(cand, np.int64))

    def joint(self, Q, qpos, pages, cand):
        """Eq. (11): greedy joint test over ``cand`` (indices into ``pages``)."""
        K, V, pos = self._layer()
        return O.joint_test(K, V, pos, Q, qpos, self.ranges(pages), list(cand),
                            tau_joint=self.th["tau_joint"], method=self.method,
                            gate="no_joint" not in self.ablation)

    def retire(self, pages):
        """L6: D_c <- D_c u A."""
        for p in pages:
            if p not in self.retired:
                self.retired.append(p)
        self.retired.sort()

    def end_commit(self):
        self.pending = None

    def post(self, Q, qpos):
        m = self.post_measure(Q, qpos)
        if len(m["cand"]):
            acc, ur = self.joint(Q, qpos, m["pages"], m["cand"])
        else:
            acc, ur = np.zeros(0, bool), np.zeros(0)
        self.retire([m["pages"][c] for c, a in zip(m["cand"], acc) if a])
        self.end_commit()
        m.update(accepted=acc, union_R=ur)
        return m

    def base_score(self, Q, qpos):
        """L5: token mass of the window, pooled (reading R12) when pool_kernel > 1."""
        K, V, pos = self._layer()
        m = O.token_mass(K, V, pos, Q, qpos)
        if self.pool[0] > 1:
            m = O.pool_scores(m, *self.pool)
        return m

    def checkpoint_lists(self):
        """L4, L6: (protectable pending pages with their R^-, retired pages
        with resident tokens as resident index ranges)."""
        pend, r = [], []
        if self.pending is not None and "no_protection" not in self.ablation \
                and "no_lifecycle" not in self.ablation:
            for p, rv in zip(*self.pending):
                if self.fully_resident(p):
                    pend.append(p)
                    r.append(rv)
        ret = []
        if "no_lifecycle" not in self.ablation:
            for p in self.retired:
                i0, i1 = self.span(p)
                if i1 > i0:
                    ret.append((i0, i1 - i0))
        return pend, np.asarray(r, np.float64), ret

    def checkpoint(self, Q, qpos, score=None):
        """Compression checkpoint (Eq. (12)-(13), Eq. (4)); L5.  ``score``
        replaces the base score (float32 per resident token) when given."""
        S = self.pos.size
        pend, r_pre, ret = self.checkpoint_lists()
        if S <= self.B and not ret:
            return dict(compacted=False)
        if score is None:
            score = self.base_score(Q, qpos)
        prng = self.ranges(pend)
        prot_idx = O.protect_pending([s for s, _ in prng], [l for _, l in prng], r_pre, self.B,
                                     self.eta, self.max_pending)
        st = O.token_states(S, ret, [prng[i] for i in prot_idx], self.keep_recent)
        keep = O.select_tokens(score, st, self.B)
        for l in range(len(self.K)):
            self.K[l], self.V[l], _ = O.compact(self.K[l], self.V[l], self.pos, keep)
        self.pos = self.pos[keep]
        self.retired = [p for p in self.retired if self.span(p)[1] > self.span(p)[0]]
        return dict(compacted=True, kept=keep, score=score, state=st,
                    protected=[pend[i] for i in prot_idx])
