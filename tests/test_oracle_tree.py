"""Pins of tree verification (oracle.tree).

* Tree-masked attention: a chain tree reduces to the chain oracle
  (oracle.attention, pinned on its own), and any tree agrees with torch's CPU
  scaled_dot_product_attention in float64 given the ancestor mask.
* Acceptance: the output law is integrated exactly over the draws (each
  child's test compares u with a threshold fixed by the tree; the final draw
  with the CDF points of the finitely many distributions it can use).  The
  emitted sequence, extended with exact target samples, must follow the
  target's joint law (brute force over a vocabulary of 5 and a tree of depth 2
  with two candidates per node, drawn as the top-2 of a draft distribution);
  the root's acceptance probability equals the target mass of its candidate
  set; planted mistakes in copies of the oracle fail the pin.
"""

import inspect
import itertools
import textwrap
from collections import defaultdict

import numpy as np
import pytest
import torch

import oracle.tree as tree_mod
from oracle import verify_attention
from oracle.tree import accept_tree, accept_tree_request, ancestor_masks, tree_attention

V5 = 5


def test_ancestor_masks_of_chain_and_star():
    chain = ancestor_masks([-1, 0, 1, 2])
    assert [int(m) for m in chain] == [0b1, 0b11, 0b111, 0b1111, 0b11111]
    star = ancestor_masks([-1, -1, -1])
    assert [int(m) for m in star] == [0b1, 0b11, 0b101, 0b1001]
    t = ancestor_masks([-1, -1, 0, 0, 1])
    assert int(t[5]) == 0b100101  # node 4 -> node 1 -> root
    with pytest.raises(ValueError):
        ancestor_masks([-1, 3, 0])


def _cache(rng, B, G, Hkv, D, lens):
    offs, tot = [], 0
    for L in lens:
        offs.append(tot)
        tot += Hkv * L * D
    k = rng.standard_normal(tot).astype(np.float32)
    v = rng.standard_normal(tot).astype(np.float32)
    return k, v, np.array(offs, dtype=np.int64), np.array(lens, dtype=np.int32)


def test_chain_tree_attention_is_chain_attention():
    rng = np.random.default_rng(1)
    B, N, Hq, Hkv, D = 2, 4, 4, 2, 16
    G = N + 1
    k, v, off, lens = _cache(rng, B, G, Hkv, D, [9, 40])
    q = rng.standard_normal((B, G, Hq, D)).astype(np.float32)
    parent = np.tile(np.arange(-1, N - 1), (B, 1))
    a = tree_attention(q, k, v, off, lens, Hkv, parent)
    b = verify_attention(q, k, v, off, lens, Hkv)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-12)


def test_tree_attention_matches_torch_sdpa_with_mask():
    rng = np.random.default_rng(2)
    B, N, Hq, Hkv, D = 2, 6, 4, 1, 8
    G = N + 1
    k, v, off, lens = _cache(rng, B, G, Hkv, D, [7, 30])
    q = rng.standard_normal((B, G, Hq, D)).astype(np.float32)
    parent = np.array([[-1, -1, 0, 0, 1, 4], [-1, 0, 0, 2, -1, 4]])
    got = tree_attention(q, k, v, off, lens, Hkv, parent)
    for b in range(B):
        L = int(lens[b])
        K = torch.from_numpy(k[off[b]:off[b] + Hkv * L * D].reshape(Hkv, L, D).astype(np.float64))
        Vv = torch.from_numpy(v[off[b]:off[b] + Hkv * L * D].reshape(Hkv, L, D).astype(np.float64))
        masks = ancestor_masks(parent[b])
        allow = torch.zeros(G, L, dtype=torch.bool)
        allow[:, :L - G] = True
        for g in range(G):
            for a in range(G):
                allow[g, L - G + a] = bool((int(masks[g]) >> a) & 1)
        Q = torch.from_numpy(q[b].astype(np.float64)).permute(1, 0, 2)          # [Hq][G][D]
        ref = torch.nn.functional.scaled_dot_product_attention(Q, K.expand(Hq, L, D), Vv.expand(Hq, L, D),
                                                               attn_mask=allow)
        np.testing.assert_allclose(got[b], ref.permute(1, 0, 2).numpy(), rtol=1e-10, atol=1e-12)


# ---- exact law of the tree acceptance --------------------------------------------

def _thresholds(p_rows, tokens, parent):
    """The fixed test threshold of every node, and the final distributions."""
    G, V = p_rows.shape
    N = G - 1
    thr = np.zeros(N)
    finals = []
    kids = [[] for _ in range(G)]
    for i in range(N):
        kids[int(parent[i]) + 1].append(i)
    for pos in range(G):
        mass, seen = 0.0, []
        for c in kids[pos]:
            t = int(tokens[c])
            thr[c] = 0.0 if t in seen else p_rows[pos][t] / (1.0 - mass)
            if t not in seen:
                mass += p_rows[pos][t]
                seen.append(t)
        r = p_rows[pos].copy()
        r[seen] = 0.0
        finals.append(r)
        finals.append(p_rows[pos])
    return thr, finals


def exact_tree_law(fn, p_rows, tokens, parent):
    p_rows = np.asarray(p_rows, dtype=np.float64)
    G, V = p_rows.shape
    N = G - 1
    thr, finals = _thresholds(p_rows, tokens, parent)
    axes = []
    for i in range(N):
        # The threshold of the algorithm, and the candidate's own probability
        # (a superset of cuts, so that variants comparing with it integrate
        # exactly too; extra cuts only subdivide).
        raw = float(p_rows[int(parent[i]) + 1][int(tokens[i])])
        cuts = {0.0, 1.0} | {x for x in (float(thr[i]), raw) if 0.0 < x < 1.0}
        axes.append(sorted(cuts))
    fc = {0.0, 1.0}
    for r in finals:
        z = r.sum()
        if z > 0:
            for x in np.cumsum(r) / z:
                if 0.0 < x < 1.0:
                    fc.add(float(x))
    axes.append(sorted(fc))
    cells = [[((a + b) / 2, b - a) for a, b in zip(c[:-1], c[1:]) if b > a] for c in axes]
    law = defaultdict(float)
    for combo in itertools.product(*cells):
        u = np.array([c[0] for c in combo])
        w = float(np.prod([c[1] for c in combo]))
        path, emitted, _, _ = fn(p_rows, tokens, parent, u)
        law[tuple(emitted)] += w
    return dict(law)


def _problem(seed):
    """Target tables over V5 tokens for depth <= 3 prefixes, and a depth-2 tree
    with the top-2 candidates of a draft distribution at each node."""
    rng = np.random.default_rng(seed)

    def dist(zeros=0):
        p = rng.dirichlet(np.ones(V5) * 0.8)
        if zeros:
            p[rng.choice(V5, size=zeros, replace=False)] = 0.0
            p /= p.sum()
        return p

    target = {(): dist(1)}
    for a in range(V5):
        target[(a,)] = dist(a % 2)
        for b in range(V5):
            target[(a, b)] = dist((a + b) % 2)

    def top2(prefix):
        q = dist()
        return [int(i) for i in np.argsort(-q, kind="stable")[:2]]

    tokens, parent, prefixes = [], [], [()]
    for t in top2(()):                       # depth 1: nodes 0, 1
        tokens.append(t)
        parent.append(-1)
        prefixes.append((t,))
    for d1 in range(2):                      # depth 2: two children per depth-1 node
        for t in top2(prefixes[d1 + 1]):
            tokens.append(t)
            parent.append(d1)
            prefixes.append(prefixes[d1 + 1] + (t,))
    p_rows = np.stack([target[pf] for pf in prefixes])
    return target, np.array(tokens), np.array(parent), p_rows


def _joint_after(fn, target, tokens, parent, p_rows, length=3):
    joint = defaultdict(float)
    for emitted, pr in exact_tree_law(fn, p_rows, tokens, parent).items():
        seqs = [(tuple(emitted), pr)]
        for k in range(len(emitted), length):
            nxt = []
            for s, m in seqs:
                row = target[s[:k]]
                for v in range(V5):
                    if row[v] > 0:
                        nxt.append((s + (v,), m * row[v]))
            seqs = nxt
        for s, m in seqs:
            joint[s[:length]] += m
    return joint


def _target_joint(target, length=3):
    out = {}
    for s in itertools.product(range(V5), repeat=length):
        out[s] = target[()][s[0]] * target[(s[0],)][s[1]] * target[s[:2]][s[2]]
    return out


@pytest.mark.parametrize("seed", [3, 4, 5])
def test_tree_verification_is_lossless(seed):
    target, tokens, parent, p_rows = _problem(seed)
    joint = _joint_after(accept_tree_request, target, tokens, parent, p_rows)
    want = _target_joint(target)
    err = max(abs(joint.get(s, 0.0) - want[s]) for s in want)
    assert err < 1e-12 and abs(sum(joint.values()) - 1.0) < 1e-12


def test_root_acceptance_is_candidate_mass():
    target, tokens, parent, p_rows = _problem(6)
    law = exact_tree_law(accept_tree_request, p_rows, tokens, parent)
    accepted_root = sum(pr for emitted, pr in law.items() if len(emitted) >= 2)
    root_kids = [int(tokens[i]) for i in range(len(parent)) if parent[i] == -1]
    assert abs(accepted_root - p_rows[0][root_kids].sum()) < 1e-12


def test_candidates_covering_the_target_always_pass():
    p_rows = np.array([[0.6, 0.4, 0.0], [0.2, 0.3, 0.5], [1.0, 0.0, 0.0]])
    law = exact_tree_law(accept_tree_request, p_rows, np.array([1, 0]), np.array([-1, -1]))
    assert abs(sum(pr for e, pr in law.items() if len(e) == 2) - 1.0) < 1e-12


def test_batched_call_and_cache_length():
    rng = np.random.default_rng(8)
    B, N, V = 5, 4, 7
    G = N + 1
    logits = rng.standard_normal((B * G, V)).astype(np.float32)
    lse = np.log(np.exp(logits.astype(np.float64)).sum(axis=1)).astype(np.float32)
    tokens = rng.integers(0, V, (B, N))
    parent = np.tile(np.array([-1, -1, 0, 2]), (B, 1))
    u = rng.random((B, G)).astype(np.float32)
    out = accept_tree(logits, lse, tokens, parent, u, kv_len=np.full(B, 50))
    for b in range(B):
        l = out["accept_len"][b]
        path = out["out_node"][b, :l]
        assert all(parent[b][path[0]] == -1 for _ in [0] if l > 0)
        for a, c in zip(path[:-1], path[1:]):
            assert parent[b][c] == a
        assert out["new_kv_len"][b] == 50 - N + l
        assert out["out_tok"][b, l] >= 0 and np.all(out["out_tok"][b, l + 1:] == -1)


_MUTATIONS = {
    "no_renormalisation": ("thr = p[t] / rest if rest > 0.0 else 0.0", "thr = p[t]"),
    "final_from_full_p": ("        r[rejected_tok] = 0.0\n", "        pass\n"),
    "longest_path_style": ("            if float(u[c]) < thr:", "            if float(u[c]) < p[int(tokens[c])] if 0 <= int(tokens[c]) < V else False:"),
    "siblings_share_draw": ("tests.append((float(u[c]), thr))\n            if float(u[c]) < thr:",
                            "tests.append((float(u[pos]), thr))\n            if float(u[pos]) < thr:"),
}


def _mutant(name):
    old, new = _MUTATIONS[name]
    src = textwrap.dedent(inspect.getsource(tree_mod.accept_tree_request))
    assert old in src, name
    ns = dict(vars(tree_mod))
    exec(compile(src.replace(old, new), "<mutant>", "exec"), ns)
    return ns["accept_tree_request"]


@pytest.mark.parametrize("name", sorted(_MUTATIONS))
def test_pin_rejects_planted_mistake(name):
    fn = _mutant(name)
    target, tokens, parent, p_rows = _problem(3)
    try:
        joint = _joint_after(fn, target, tokens, parent, p_rows)
    except Exception:
        return
    want = _target_joint(target)
    err = max(abs(joint.get(s, 0.0) - want[s]) for s in want)
    assert err > 1e-6, f"pin did not catch {name}"


def test_commit_keeps_a_chain_in_place_and_compacts_a_path():
    from oracle.tree import tree_commit_kv
    D, Hkv, N = 4, 2, 5
    L = 9
    k = np.arange(Hkv * L * D, dtype=np.float32)
    v = -k
    same_k, same_v = tree_commit_kv(k, v, [0], [L], Hkv, D, [[0, 1, 2, -1, -1, -1]], [3], N)
    assert np.array_equal(same_k, k) and np.array_equal(same_v, v)     # a chain prefix is already in place
    got_k, _ = tree_commit_kv(k, v, [0], [L], Hkv, D, [[1, 3, -1, -1, -1, -1]], [2], N)
    tail0 = L - (N + 1)
    for g in range(Hkv):
        rows = got_k[g * L * D:(g + 1) * L * D].reshape(L, D)
        orig = k[g * L * D:(g + 1) * L * D].reshape(L, D)
        assert np.array_equal(rows[tail0 + 1], orig[tail0 + 2])        # node 1
        assert np.array_equal(rows[tail0 + 2], orig[tail0 + 4])        # node 3
        assert np.array_equal(rows[:tail0 + 1], orig[:tail0 + 1])      # prefix and root untouched
