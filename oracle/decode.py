"""Image decode with draft-then-verify cycles, and the plain AR reference.

A cycle (Sec. 3.1): the draft head proposes a tree of depth d and width k chosen by the
ADT rule (Sec. 4), the target verifies every node in one forward under the tree mask,
the longest acceptable root-to-node path plus one bonus token is committed, and the
caches are compacted so that the accepted nodes' K/V become the next prefix.

State conventions (the paper gives none):
  * the root of a tree is the last committed token; its target K/V are not cached yet,
    so the target cache holds L = (committed tokens - 1) positions;
  * tree node i is verified at position L + depth(i) and its K/V go to slot L + i;
    compaction copies slot L + v_m to slot L + m for the accepted nodes v_1 < .. < v_a;
  * the draft row of the token at position p takes the target feature of position p-1
    (zeros before position 0); a tree node whose parent is not committed takes the draft
    feature of its parent's row instead, the root's draft row standing in for the root;
  * each cycle first runs the draft head over the tokens committed by the previous cycle
    (catch-up rows, the root last), then d - 1 forwards over the frontier.

Test infrastructure only; see the package docstring.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

from synth import DecodeCfg
from . import accept as acc
from .attention import tree_key_slots
from .expand import Tree, build_tree, expand, expand_sampled
from .model import OracleModel
from .numerics import draw_below, masked_logits, uniform_u64
from .schedule import initial, schedule
from .tree import ancestors_and_self


@dataclasses.dataclass
class StepInfo:
    step: int
    d_hat: int
    k_hat: int
    tree: Tree
    logits: np.ndarray          # [n][V] verify logits (allowed-range masking not applied)
    allowed: np.ndarray         # [n][2] allowed id range of the token each row predicts
    path: List[int]             # accepted node indices v_1..v_a
    bonus: int
    committed: List[int]        # tokens committed this cycle
    L_before: int
    draft_root_logits: Optional[np.ndarray] = None


def compact_cache(k: np.ndarray, v: np.ndarray, L: int, path: List[int]) -> None:
    """KV compaction: the accepted nodes v_1 < .. < v_a take cache slots L+1 .. L+a (slot axis
    is the second to last), in order, so that they become the committed prefix."""
    for m, node in enumerate(path, start=1):
        k[..., L + m, :] = k[..., L + node, :]
        v[..., L + m, :] = v[..., L + node, :]


class Branch:
    """One guidance branch (Sec. 3.1, CFG): its own prompt, target and draft caches and
    target features; the image tokens are shared by all branches."""

    def __init__(self, model: OracleModel, prefix, s_cap: int):
        self.prefix = [int(t) for t in prefix]
        self.tcache, self.dcache = model.new_caches(s_cap)
        self.feat: Dict[int, np.ndarray] = {}          # target feature per committed position


def guide(rows: List[np.ndarray], scale: Optional[float]) -> np.ndarray:
    """Classifier-free guidance (Ho & Salimans) on logits: l_u + s (l_c - l_u); one branch
    passes through."""
    if scale is None:
        return rows[0]
    cond, uncond = rows
    return uncond + scale * (cond - uncond)


class Decoder:
    """Oracle decode state for one image."""

    def __init__(self, cfg: DecodeCfg, model: OracleModel, prefix: np.ndarray,
                 poisson: Optional[np.ndarray] = None, knn: Optional[np.ndarray] = None,
                 accept_seed: Optional[int] = None, uncond_prefix: Optional[np.ndarray] = None):
        self.cfg = cfg
        self.model = model
        self.P = len(prefix)
        self.tokens: List[int] = [int(t) for t in prefix]
        s_cap = self.P + cfg.n_image + 256
        self.guidance = cfg.guidance
        prompts = [prefix]
        if cfg.guidance is not None:
            assert uncond_prefix is not None and len(uncond_prefix) == self.P
            prompts.append(uncond_prefix)
        self.branches = [Branch(model, pr, s_cap) for pr in prompts]
        self.records: Dict[int, Tuple[int, int]] = {}  # cell -> (d, k) of the committing tree
        self.prev: Optional[Tuple[int, int]] = None    # (a, d) of the previous tree
        self.prev_cell: Optional[int] = None
        self.L = 0
        self.Ld = 0
        self.step_no = 0
        self.poisson = poisson
        self.knn = knn
        self.accept_seed = cfg.seed if accept_seed is None else accept_seed
        self.q_rows: Dict[int, np.ndarray] = {}   # stochastic children: tree index -> draft row of its children

    # the conditional (or only) branch's state
    @property
    def tcache(self):
        return self.branches[0].tcache

    @property
    def dcache(self):
        return self.branches[0].dcache

    @property
    def feat(self):
        return self.branches[0].feat

    # ---------------------------------------------------------------- helpers
    def allowed_pos(self, p: int) -> Tuple[int, int]:
        """Allowed id range of the token at absolute position p (an image position)."""
        return self.cfg.allowed(p - self.P)

    def committed_image(self) -> int:
        return len(self.tokens) - self.P

    def done(self) -> bool:
        return self.committed_image() >= self.cfg.n_image

    def _pick(self, logit_rows: np.ndarray, parent, token, allowed, step: int):
        a = self.cfg.accept
        if a.mode == "greedy":
            return acc.accept_greedy(logit_rows, parent, token, allowed)
        if a.mode == "mss":
            return acc.accept_mss(logit_rows, self.q_rows, parent, token, allowed, temperature=a.temperature,
                                  top_k=a.top_k, seed=self.accept_seed, step=step)
        return acc.accept_sampling(logit_rows, parent, token, allowed, temperature=a.temperature,
                                   top_k=a.top_k, seed=self.accept_seed, step=step, mode=a.mode,
                                   delta=a.delta, knn=self.knn, knn_k=a.knn_k)

    def _feat_before(self, br: Branch, p: int) -> np.ndarray:
        return br.feat[p - 1] if p > 0 else np.zeros(self.cfg.model.d_model)

    # ---------------------------------------------------------------- prefill
    def prefill(self) -> int:
        """Target and draft over each branch's prompt, then the first image token by one AR
        step on the (guided) logits of the last prompt row."""
        P = self.P
        pos = list(range(P))
        causal = [list(range(r + 1)) for r in range(P)]
        last = []
        for br in self.branches:
            logits, f = self.model.target_rows(br.prefix, pos, pos, causal, br.tcache)
            for p in range(P):
                br.feat[p] = f[p]
            par = np.stack([self._feat_before(br, p) for p in range(P)])
            self.model.draft_rows(br.prefix, par, pos, pos, causal, br.dcache)
            last.append(logits[P - 1])
        lo, hi = self.allowed_pos(P)
        self.prefill_branch_logits = last
        self.prefill_logits = guide(last, self.guidance)
        _, first = self._pick(self.prefill_logits[None], [-1], [self.tokens[-1]], np.array([[lo, hi]]), 0)
        self.tokens.append(first)
        self.L = P
        self.Ld = P
        self.step_no = 1
        return first

    # ---------------------------------------------------------------- draft side
    def _draft_catch_up(self):
        """Draft rows for committed positions Ld..L (the root last), every branch.  Returns
        the root row's guided logits and its draft feature per branch."""
        ps = list(range(self.Ld, self.L + 1))
        toks = [self.tokens[p] for p in ps]
        keys = [list(range(p + 1)) for p in ps]
        lgs, feats = [], []
        for br in self.branches:
            par = np.stack([self._feat_before(br, p) for p in ps])
            lg, fd = self.model.draft_rows(toks, par, ps, ps, keys, br.dcache)
            lgs.append(lg[-1])
            feats.append(fd[-1])
        self.draft_root_branch_logits = lgs
        return guide(lgs, self.guidance), feats

    def expand_tree(self, d_hat: int, k_hat: int):
        L = self.L
        root_logits, root_feat = self._draft_catch_up()
        row_slot: Dict[int, int] = {}       # pool index -> draft cache slot of its row
        row_feat: Dict[int, List[np.ndarray]] = {}   # pool index -> draft feature per branch
        next_slot = [L + 1]

        def level_fn(frontier, pool):
            toks, pos, slots, keys = [], [], [], []
            for u in frontier:
                node = pool[u]
                toks.append(node.token)
                pos.append(L + node.depth)
                slot = next_slot[0]
                next_slot[0] += 1
                row_slot[u] = slot
                slots.append(slot)
                anc = []
                v = node.parent
                while v != -1:
                    anc.append(row_slot[v])
                    v = pool[v].parent
                keys.append(list(range(L + 1)) + sorted(anc) + [slot])
            lgs = []
            for b, br in enumerate(self.branches):
                feats = [root_feat[b] if pool[u].parent == -1 else row_feat[pool[u].parent][b] for u in frontier]
                lg, fd = self.model.draft_rows(toks, np.stack(feats), pos, slots, keys, br.dcache)
                for u, frow in zip(frontier, fd):
                    row_feat.setdefault(u, []).append(frow)
                lgs.append(lg)
            return guide(lgs, self.guidance)

        a = self.cfg.accept
        allowed_at = lambda depth: self.allowed_pos(L + depth)
        if a.mode == "mss":
            # stochastic children: q of every expanded node is kept for the acceptance, keyed by
            # the node's tree index (pool index + 1; the root is 0)
            self.q_rows = {0: root_logits}

            def sampled_level(frontier, pool):
                rows = level_fn(frontier, pool)
                for u, row in zip(frontier, rows):
                    self.q_rows[u + 1] = row
                return rows

            pool, sel = expand_sampled(root_logits, sampled_level, d_hat, k_hat, a.children, self.cfg.sched.n_budget,
                                       allowed_at, temperature=a.temperature, top_k=a.top_k, seed=self.accept_seed,
                                       step=self.step_no)
            return build_tree(self.tokens[-1], pool, sel, by_creation=True), root_logits
        pool, sel = expand(root_logits, level_fn, d_hat, k_hat, self.cfg.sched.n_budget, allowed_at)
        return build_tree(self.tokens[-1], pool, sel), root_logits

    # ---------------------------------------------------------------- one cycle
    def verify(self, tree: Tree):
        """Target forward of every tree node in each branch.  Returns (guided logits,
        features per branch, allowed ranges); the per-branch logits stay in
        self.verify_branch_logits."""
        L = self.L
        anc = ancestors_and_self(tree.parent)
        pos = [L + int(dp) for dp in tree.depth]
        slots = [L + i for i in range(tree.n)]
        lgs, fs = [], []
        for br in self.branches:
            logits, f = self.model.target_rows(tree.token, pos, slots, tree_key_slots(L, anc), br.tcache)
            lgs.append(logits)
            fs.append(f)
        self.verify_branch_logits = lgs
        allowed = np.array([self.allowed_pos(L + int(dp) + 1) for dp in tree.depth], dtype=np.int64)
        return guide(lgs, self.guidance), fs, allowed

    def schedule_next(self) -> Tuple[int, int]:
        cell = self.L + 1 - self.P                   # cell of the first drafted token
        remaining = self.cfg.n_image - cell
        prev = self.prev
        if prev is not None and self.cfg.sched.alpha_source == "poisson" and self.poisson is not None:
            prev = (min(int(self.poisson[self.prev_cell]), prev[1]), prev[1])
        init = initial(self.cfg.sched, cell, self.records, self.cfg.grid_w)
        return schedule(self.cfg.sched, init, prev, remaining)

    def compact(self, path: List[int]):
        for br in self.branches:
            compact_cache(br.tcache.k, br.tcache.v, self.L, path)

    def step(self) -> StepInfo:
        d_hat, k_hat = self.schedule_next()
        if d_hat >= 1:
            tree, draft_root = self.expand_tree(d_hat, k_hat)
            return self.verify_commit(tree, d_hat, k_hat, expanded=True, draft_root=draft_root)
        return self.verify_commit(build_tree(self.tokens[-1], [], []), d_hat, k_hat, expanded=False)

    def verify_commit(self, tree: Tree, d_hat: int, k_hat: int, expanded: bool = False,
                      draft_root: Optional[np.ndarray] = None) -> StepInfo:
        """Verify a tree, accept along it, compact and commit.  Without a preceding expansion
        (expanded=False) the draft cache was not advanced, so its valid length stays."""
        L = self.L
        logits, fs, allowed = self.verify(tree)
        masked = np.stack([masked_logits(logits[i], *allowed[i]) for i in range(tree.n)])
        path, bonus = self._pick(masked, tree.parent, tree.token, allowed, self.step_no)
        committed = [int(tree.token[v]) for v in path] + [int(bonus)]
        self.compact(path)
        for br, f in zip(self.branches, fs):
            br.feat[L] = f[0]
            for m, v in enumerate(path, start=1):
                br.feat[L + m] = f[v]
        cell0 = L + 1 - self.P
        for c in range(cell0, cell0 + len(committed)):
            self.records[c] = (d_hat, k_hat)
        self.prev = (len(path), d_hat)
        self.prev_cell = cell0
        self.tokens += committed
        if expanded:
            self.Ld = L + 1
        self.L = L + 1 + len(path)
        info = StepInfo(self.step_no, d_hat, k_hat, tree, logits, allowed, path, int(bonus), committed, L,
                        draft_root)
        self.step_no += 1
        return info

    def run(self, max_steps: Optional[int] = None) -> List[StepInfo]:
        out = []
        while not self.done() and (max_steps is None or len(out) < max_steps):
            out.append(self.step())
        return out


def ar_decode(cfg: DecodeCfg, model: OracleModel, prefix: np.ndarray, n_tokens: Optional[int] = None,
              uncond_prefix: Optional[np.ndarray] = None):
    """Plain greedy AR reference: prefill, then one target row per token (per guidance
    branch, the logits combined by CFG).  Returns (image tokens, per-token guided logits of
    the row that predicted each token after the first)."""
    assert cfg.accept.mode == "greedy"
    prompts = [prefix] if cfg.guidance is None else [prefix, uncond_prefix]
    P = len(prefix)
    n_tokens = cfg.n_image if n_tokens is None else n_tokens
    caches = [model.new_caches(P + n_tokens + 1)[0] for _ in prompts]
    pos = list(range(P))
    causal = [list(range(r + 1)) for r in range(P)]
    last = [model.target_rows([int(t) for t in pr], pos, pos, causal, c)[0][P - 1] for pr, c in zip(prompts, caches)]
    g = guide(last, cfg.guidance)
    lo, hi = cfg.allowed(0)
    toks = [lo + int(np.argmax(g[lo:hi]))]
    rows = []
    for i in range(1, n_tokens):
        p = P + i - 1                                  # position of the latest token
        g = guide([model.target_rows([toks[-1]], [p], [p], [list(range(p + 1))], c)[0][0] for c in caches],
                  cfg.guidance)
        rows.append(g)
        lo, hi = cfg.allowed(i)
        toks.append(lo + int(np.argmax(g[lo:hi])))
    return toks, rows
