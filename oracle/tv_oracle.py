"""Literal float64 Traversal Verification and token-level verification.

TEST INFRASTRUCTURE ONLY: imported by tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py, never by the library.

Every step follows the paper (arXiv 2505.12398) in its own order and notation,
with whole probability vectors over the vocabulary held and updated eagerly:

* Algorithm 3 (Sec. 3.1): initialise p^ini along every chain, then repeatedly
  take the chain from the root to the first leaf of the remaining tree, test its
  leaf, and on rejection delete the leaf and update its parent with Eq. (e1)
  (residual target), Eq. (e2) (draft with the rejected token removed) and
  Eq. (e3) (parent acceptance rate), then re-rate every remaining chain through
  that parent. Finally sample Y from the (possibly residual) target at X^tau.
* Token-level tree verification (Sec. 2.2): layer by layer from the root, the
  children of the current node are verified with recursive rejection sampling
  (Algorithm 2, with the zero-and-renormalise draft step in the
  without-replacement case); an accepted child becomes the current node.

Conventions where the paper leaves a choice open (each is listed with its
reason in the design notes):

* children are ordered by ascending node index; nodes are numbered so that
  parent[i] < i; "the first leaf" is reached through first children
  (post-order DFS, App. E);
* row i of the logits is the next-token distribution after the path root..i;
  a child's ratio uses its parent's rows;
* uniforms: u[i] tests node i, u[0] drives the final sample; accept iff u < theta;
* the final sample is an inverse CDF in ascending token order with
  y = min{y : u*W < C(y)}, C the running sum and W = C(V-1);
* sibling mode: WITHOUT_REPLACEMENT uses Eq. (e2) (the paper's default, valid for
  children drawn without replacement); WITH_REPLACEMENT leaves the draft
  distribution unchanged after a rejection (children drawn i.i.d.);
* a non-root parent whose residual mass S is exactly zero gets p = 0 (the Sec. 3.2
  example drops such a node at once, since it can never be accepted); its
  remaining descendants are PRUNED: they are not tested and their rejection
  triggers no update;
* a residual mass of zero where the algorithm needs a residual distribution
  (the root in Algorithm 3, any node in the token-level algorithm) cannot occur
  in exact arithmetic; if rounding produces it the tree reports DEGENERATE.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

WITHOUT_REPLACEMENT = 0
WITH_REPLACEMENT = 1

TREE_OK = 0
TREE_BAD_PARENT = 1
TREE_BAD_TOKEN = 2
TREE_DUP_SIBLING = 3
TREE_NONFINITE = 4
TREE_DEGENERATE = 5

NODE_UNTESTED = 0
NODE_ACCEPTED = 1
NODE_REJECTED = 2
NODE_PRUNED = 3


@dataclass
class TreeResult:
    status: int
    accept_len: int = -1          # tau: depth of the accepted node
    accepted_node: int = -1       # X^tau ends at this node; the path is its ancestors
    bonus_token: int = -1         # Y
    node_state: np.ndarray = None  # int8 [N+1]
    node_theta: np.ndarray = None  # float64 [N+1]; -1 where untested, 0 where pruned
    p_init: np.ndarray = None      # float64 [N+1]; Alg. 3 initialisation
    rows_consulted: int = 0        # internal nodes that are proper ancestors of a tested node
    residual_passes: int = 0       # Eq. (e1)-(e3) updates executed
    leaf_accepted: int = 0         # 1 if the accepted node has no children in the input tree
    tests: int = 0                 # nodes compared against a uniform
    # Early rejection (bookkeeping for verifiers that skip updates that decide
    # nothing): a rejection that removes the last remaining child of a non-root
    # node j while u[j] >= p(j) needs no update at j, since Eq. (e3) never
    # raises p(j) (S <= p(j) by Eq. (e1)), so j is rejected whatever S is.
    early_rejections: int = 0      # updates a verifier with early rejection skips
    early_margin: float = float("inf")  # min |u[j] - p(j)| over the rule's checks
    early_nodes: list = field(default_factory=list)  # the j of each skipped update
    test_order: list = field(default_factory=list)
    margins: dict = field(default_factory=dict)   # node -> |u - theta| for tested nodes
    y_weights: np.ndarray = None   # distribution Y is drawn from
    y_margin: float = float("inf")  # distance of u*W to the nearest CDF boundary, / W

    @property
    def counters(self):
        return (self.rows_consulted, self.residual_passes, self.leaf_accepted, self.tests)

    @property
    def counters_early(self):
        """Counters of a verifier that applies early rejection: the same, with
        only the residual updates it executes."""
        return (self.rows_consulted, self.residual_passes - self.early_rejections,
                self.leaf_accepted, self.tests)


# ---------------------------------------------------------------------------
# Input handling
# ---------------------------------------------------------------------------

def to_f64(logits) -> np.ndarray:
    """Exact float64 copy of logits. bfloat16 arrives as its uint16 bit pattern
    and is widened exactly (the 16 bits become the top half of a float32)."""
    a = np.asarray(logits)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def tempered_softmax(z, T: float) -> np.ndarray:
    """softmax(z / T) in float64: the distributions M_b(.|X^i) and M_s(.|X^i) of
    the problem statement (Alg. 3, REQUIRE) at sampling temperature T > 0
    (Sec. 4.4; App. H requires T > 0). Returns None if the row has NaN or +inf
    or no finite entry."""
    z = np.asarray(z, dtype=np.float64)
    if np.isnan(z).any() or np.isposinf(z).any():
        return None
    m = z.max()
    if not np.isfinite(m):
        return None
    e = np.exp((z - m) / T)
    return e / e.sum()


def _structure(parents, tokens, V, mode):
    """Validate the tree and build child lists in ascending index order.
    Returns (status, children, depth)."""
    n1 = len(parents)
    if n1 < 1 or int(parents[0]) != -1:
        return TREE_BAD_PARENT, None, None
    for i in range(1, n1):
        if not 0 <= int(parents[i]) < i:
            return TREE_BAD_PARENT, None, None
    for i in range(1, n1):
        if not 0 <= int(tokens[i]) < V:
            return TREE_BAD_TOKEN, None, None
    children = [[] for _ in range(n1)]
    depth = [0] * n1
    for i in range(1, n1):
        children[int(parents[i])].append(i)
        depth[i] = depth[int(parents[i])] + 1
    if mode == WITHOUT_REPLACEMENT:
        for j in range(n1):
            toks = [int(tokens[c]) for c in children[j]]
            if len(set(toks)) != len(toks):
                return TREE_DUP_SIBLING, None, None
    return TREE_OK, children, depth


# ---------------------------------------------------------------------------
# The paper's update steps, one function each
# ---------------------------------------------------------------------------

def chain_rate(p_parent: float, b_parent: np.ndarray, s_parent: np.ndarray, x: int) -> float:
    """Acceptance rate of a chain extended by token x (Alg. 3 initialisation and
    re-rating step): min(p(parent) * M_b(x|parent) / M_s(x|parent), 1). A zero
    numerator gives rate 0 whatever the draft holds."""
    if p_parent == 0.0 or b_parent[x] == 0.0:
        return 0.0
    return min(p_parent * b_parent[x] / s_parent[x], 1.0)


def residual_e1(p_parent: float, b: np.ndarray, s: np.ndarray):
    """Eq. (e1): unnormalised residual [p * M_b - M_s]_+ and its mass S (the sum
    that also appears in Eq. (e3))."""
    d = np.maximum(p_parent * b - s, 0.0)
    return d, float(d.sum())


def draft_update_e2(s: np.ndarray, x: int) -> np.ndarray:
    """Eq. (e2): the rejected token x gets draft probability 0 and the other
    entries are renormalised."""
    s = s.copy()
    s[x] = 0.0
    return s / s.sum()


def acceptance_update_e3(S: float, p_parent: float) -> float:
    """Eq. (e3): p' = S / (S + 1 - p), with the parent's missing mass 1 - p formed
    first (exact for p in [1/2, 1], and exactly 1 at the root where p = 1)."""
    return S / (S + (1.0 - p_parent))


def rrs_residual(b: np.ndarray, s: np.ndarray):
    """Algorithm 2, rejection branch: M_b' <- norm([M_b' - M_s']_+). Returns the
    normalised residual, or None if its mass is zero."""
    d = np.maximum(b - s, 0.0)
    S = d.sum()
    if S <= 0.0:
        return None
    return d / S


def inverse_cdf(w: np.ndarray, u: float):
    """Inverse-CDF sample in ascending token order: the smallest y with
    u*W < C(y), C the running sum of w and W = C(V-1) from the same sum.
    Returns (y, margin): margin is the distance of u*W to the nearest boundary
    of y's interval, divided by W (used to recognise near-ties)."""
    c = np.cumsum(np.asarray(w, dtype=np.float64))
    W = c[-1]
    if not W > 0.0:
        return -1, 0.0
    t = u * W
    y = int(np.searchsorted(c, t, side="right"))
    if y >= len(c):  # cannot happen for u < 1; kept for rounding safety
        y = int(np.nonzero(np.asarray(w) > 0)[0][-1])
    lo = c[y - 1] if y > 0 else 0.0
    return y, float(min(t - lo, c[y] - t) / W)


def _uniform_decider(uniforms):
    def decide(node, theta):
        return float(uniforms[node]) < theta
    return decide


def _finish(res: TreeResult, children, depth, parents, uniforms):
    """Shared bookkeeping once the accepted node and Y's distribution are known."""
    tested = [i for i in res.test_order]
    consulted = set()
    for t in tested:
        a = int(parents[t])
        while a >= 0:
            consulted.add(a)
            a = int(parents[a])
    res.rows_consulted = len(consulted)
    res.tests = len(tested)
    res.accept_len = depth[res.accepted_node]
    res.leaf_accepted = 0 if children[res.accepted_node] else 1
    if uniforms is not None and res.y_weights is not None:
        y, margin = inverse_cdf(res.y_weights, float(uniforms[0]))
        res.bonus_token = y
        res.y_margin = margin
        if y < 0:
            res.status = TREE_DEGENERATE
    return res


def _error(status, n1):
    return TreeResult(status=status,
                      node_state=np.zeros(n1, np.int8),
                      node_theta=np.full(n1, -1.0),
                      p_init=np.full(n1, -1.0))


# ---------------------------------------------------------------------------
# Algorithm 3: Traversal Verification
# ---------------------------------------------------------------------------

def _init_chains(parents, tokens, children, b, s):
    """Alg. 3 initialisation: p^ini(X_0) = 1 and, in index order (parents come
    first), p^ini(X_i) = min(p^ini(X_{i-1}) * M_b(X_i|X^{i-1}) / M_s(X_i|X^{i-1}), 1)."""
    n1 = len(parents)
    p = np.zeros(n1)
    p[0] = 1.0
    for i in range(1, n1):
        j = int(parents[i])
        p[i] = chain_rate(p[j], b[j], s[j], int(tokens[i]))
    return p


def verify_tree(parents, tokens, target_logits, draft_logits, temperature, uniforms,
                mode=WITHOUT_REPLACEMENT, decide=None) -> TreeResult:
    """Algorithm 3 on one tree.

    parents[i], tokens[i]: node i's parent (parents[0] = -1, parents[i] < i) and
    drafted token; target_logits/draft_logits: [N+1][V] rows (float64, or bf16
    bits as uint16); temperature: the float32 value used by both models;
    uniforms: [N+1] values in [0,1) (u[i] tests node i, u[0] samples Y), or None
    together with a ``decide(node, theta) -> bool`` callback (enumeration).
    """
    n1 = len(parents)
    zb = to_f64(target_logits)
    zs = to_f64(draft_logits)
    V = zb.shape[-1]
    T = float(np.float32(temperature))
    status, children, depth = _structure(parents, tokens, V, mode)
    if status != TREE_OK:
        return _error(status, n1)
    if decide is None:
        decide = _uniform_decider(uniforms)

    # Target and draft distributions of every node that has children (REQUIRE).
    b, s = {}, {}
    for j in range(n1):
        if children[j]:
            Pj = tempered_softmax(zb[j], T)
            Qj = tempered_softmax(zs[j], T)
            if Pj is None or Qj is None:
                return _error(TREE_NONFINITE, n1)
            b[j], s[j] = Pj, Qj
    for i in range(1, n1):
        if s[int(parents[i])][int(tokens[i])] == 0.0:   # token the draft cannot produce
            return _error(TREE_NONFINITE, n1)

    p = _init_chains(parents, tokens, children, b, s)
    res = TreeResult(status=TREE_OK,
                     node_state=np.zeros(n1, np.int8),
                     node_theta=np.full(n1, -1.0),
                     p_init=p.copy())
    alive = [True] * n1

    while True:
        # Select the chain from the root to the first leaf of the remaining tree.
        leaf = 0
        while True:
            nxt = next((c for c in children[leaf] if alive[c]), None)
            if nxt is None:
                break
            leaf = nxt
        if leaf == 0:                       # only the root is left: p(X_0) = 1
            res.accepted_node = 0
            if res.node_state[0] == NODE_UNTESTED:
                res.node_state[0] = NODE_ACCEPTED
            break
        j = int(parents[leaf])
        if p[j] == 0.0:                     # parent can no longer be accepted
            res.node_state[leaf] = NODE_PRUNED
            res.node_theta[leaf] = 0.0
            alive[leaf] = False
            continue
        theta = float(p[leaf])
        res.node_theta[leaf] = theta
        res.test_order.append(leaf)
        if uniforms is not None:
            res.margins[leaf] = abs(float(uniforms[leaf]) - theta)
        if decide(leaf, theta):
            res.node_state[leaf] = NODE_ACCEPTED
            res.accepted_node = leaf
            break
        res.node_state[leaf] = NODE_REJECTED
        alive[leaf] = False                 # T <- T - {X_gamma}
        if uniforms is not None:
            _early_rejection(res, children, alive, p, uniforms, j)

        # Residual and draft distributions at the parent, Eq. (e1) and (e2).
        d, S = residual_e1(p[j], b[j], s[j])
        if S > 0.0:
            b[j] = d / S
        if mode == WITHOUT_REPLACEMENT:
            s[j] = draft_update_e2(s[j], int(tokens[leaf]))
        # Parent acceptance rate, Eq. (e3).
        if S > 0.0:
            p[j] = acceptance_update_e3(S, p[j])
        elif j == 0:
            return _error(TREE_DEGENERATE, n1)
        else:
            p[j] = 0.0
        res.residual_passes += 1
        rerate_chains(p, b, s, parents, tokens, alive, j)

    acc = res.accepted_node
    if children[acc]:
        res.y_weights = b[acc]
    else:
        res.y_weights = tempered_softmax(zb[acc], T)
        if res.y_weights is None:
            return _error(TREE_NONFINITE, n1)
    return _finish(res, children, depth, parents, uniforms)


def _early_rejection(res: TreeResult, children, alive, p, uniforms, j):
    """Counts the update at j as one an early-rejecting verifier skips when j
    is not the root, j has no remaining child, and u[j] >= p(j) before the
    update. p(j) only falls under Eq. (e3): S = sum [p(j) b - s]_+ <= p(j)
    (Eq. (e1)) and S / (S + 1 - p(j)) grows with S, reaching p(j) at S = p(j).
    So j, tested next, is rejected whatever S is."""
    if j == 0 or any(alive[c] for c in children[j]):
        return
    u = float(uniforms[j])
    res.early_margin = min(res.early_margin, abs(u - float(p[j])))
    if u >= p[j]:
        res.early_rejections += 1
        res.early_nodes.append(j)


def rerate_chains(p, b, s, parents, tokens, alive, j):
    """Alg. 3 update step after a rejection: every remaining chain that passes
    through the modified node j is re-rated from j's new p, M_b and M_s (index
    order keeps each node after its own parent)."""
    for dnode in range(j + 1, len(parents)):
        if alive[dnode] and _is_descendant(parents, dnode, j):
            pd = int(parents[dnode])
            p[dnode] = chain_rate(p[pd], b[pd], s[pd], int(tokens[dnode]))


def _is_descendant(parents, d, j):
    a = int(parents[d])
    while a > j:
        a = int(parents[a])
    return a == j


# ---------------------------------------------------------------------------
# Token-level tree verification (Sec. 2.2, Algorithm 2 per node)
# ---------------------------------------------------------------------------

def verify_tree_tokenlevel(parents, tokens, target_logits, draft_logits, temperature,
                           uniforms, mode=WITHOUT_REPLACEMENT, decide=None) -> TreeResult:
    """Top-down token-level verification with recursive rejection sampling.
    Same arguments and uniform layout as :func:`verify_tree`."""
    n1 = len(parents)
    zb = to_f64(target_logits)
    zs = to_f64(draft_logits)
    V = zb.shape[-1]
    T = float(np.float32(temperature))
    status, children, depth = _structure(parents, tokens, V, mode)
    if status != TREE_OK:
        return _error(status, n1)
    if decide is None:
        decide = _uniform_decider(uniforms)

    res = TreeResult(status=TREE_OK,
                     node_state=np.zeros(n1, np.int8),
                     node_theta=np.full(n1, -1.0),
                     p_init=np.full(n1, -1.0))
    j = 0
    while True:
        if not children[j]:                 # reached a leaf: Y ~ M_b(.|X^tau)
            res.accepted_node = j
            if j == 0:
                res.node_state[0] = NODE_ACCEPTED
            res.y_weights = tempered_softmax(zb[j], T)
            if res.y_weights is None:
                return _error(TREE_NONFINITE, n1)
            break
        b = tempered_softmax(zb[j], T)      # M_b' initialised with M_b
        s = tempered_softmax(zs[j], T)      # M_s' initialised with M_s
        if b is None or s is None:
            return _error(TREE_NONFINITE, n1)
        nxt = None
        for c in children[j]:
            x = int(tokens[c])
            if s[x] == 0.0:                 # token the draft cannot produce
                return _error(TREE_NONFINITE, n1)
            theta = 0.0 if b[x] == 0.0 else min(b[x] / s[x], 1.0)
            res.node_theta[c] = theta
            res.test_order.append(c)
            if uniforms is not None:
                res.margins[c] = abs(float(uniforms[c]) - theta)
            if decide(c, theta):
                res.node_state[c] = NODE_ACCEPTED
                nxt = c
                break
            res.node_state[c] = NODE_REJECTED
            b = rrs_residual(b, s)
            if b is None:
                return _error(TREE_DEGENERATE, n1)
            if mode == WITHOUT_REPLACEMENT:
                s = draft_update_e2(s, x)
            res.residual_passes += 1
        if nxt is None:                     # every candidate rejected: Y ~ residual
            res.accepted_node = j
            res.y_weights = b
            if j == 0:
                res.node_state[0] = NODE_ACCEPTED
            break
        j = nxt
    return _finish(res, children, depth, parents, uniforms)


# ---------------------------------------------------------------------------
# The accepted output (Def. def2): the chain X^tau from the root, then Y
# ---------------------------------------------------------------------------

def committed_sequence(parents, tokens, accepted_node: int, bonus_token: int):
    """The verification output as it is committed for the next cycle: the
    nodes of the accepted chain X^tau after the root, in order from the root
    (the drafted positions whose cache entries are kept), and their tokens
    followed by Y. Returns (nodes, tokens), both lists."""
    chain = []
    x = int(accepted_node)
    while x > 0:
        chain.append(x)
        x = int(parents[x])
    chain.reverse()
    return chain, [int(tokens[c]) for c in chain] + [int(bonus_token)]
