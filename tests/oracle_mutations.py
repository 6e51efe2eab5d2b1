"""Plausible mistakes planted in the oracle (CPU only) to show that its pins
catch them.  ``tests/conftest.py`` applies one of these when the environment
variable ORACLE_MUTATION names it; ``test_oracle_mutations.py`` runs the pin
suites under each and expects a failure."""

import numpy as np

import oracle.accept as oa
import oracle.decode as od
import oracle.draft as odr
import oracle.model as om
import oracle.sampling as osm
import oracle.verify as ov

_MODULES = (om, ov, od, oa, osm, odr)


def _patch(name, fn):
    for mod in _MODULES:
        if hasattr(mod, name):
            setattr(mod, name, fn)


def rope_sign():
    def rope(x, pos, base):
        dh = x.shape[-1]
        half = dh // 2
        ang = np.asarray(pos, dtype=np.float64)[..., None] * om.rope_inv_freq(dh, base)
        c, s = np.cos(ang), np.sin(ang)
        x1, x2 = x[..., :half], x[..., half:]
        return np.concatenate([x1 * c + x2 * s, x2 * c - x1 * s], axis=-1)
    _patch("rope", rope)


def rope_interleaved():
    def rope(x, pos, base):
        dh = x.shape[-1]
        ang = np.asarray(pos, dtype=np.float64)[..., None] * om.rope_inv_freq(dh, base)
        c, s = np.cos(ang), np.sin(ang)
        x1, x2 = x[..., 0::2], x[..., 1::2]
        out = np.empty_like(x)
        out[..., 0::2] = x1 * c - x2 * s
        out[..., 1::2] = x2 * c + x1 * s
        return out
    _patch("rope", rope)


def rope_freq_exponent():
    _orig = om.rope_inv_freq
    om.rope_inv_freq = lambda dh, base: base ** (-np.arange(dh // 2, dtype=np.float64) / dh)


def rmsnorm_eps_outside():
    _patch("rmsnorm", lambda x, g, eps: x / (np.sqrt(np.mean(x * x, axis=-1, keepdims=True)) + eps) * g)


def attention_unscaled():
    def tree_attention(q, k, v, Kp, Vp, visible):
        T, Hq, dh = q.shape
        group = Hq // k.shape[1]
        o = np.zeros((T, Hq, dh))
        for hq in range(Hq):
            hk = hq // group
            keys = np.concatenate([Kp[hk], k[:, hk, :]], axis=0)
            vals = np.concatenate([Vp[hk], v[:, hk, :]], axis=0)
            s = np.where(visible, q[:, hq, :] @ keys.T, -np.inf)
            o[:, hq, :] = om.softmax(s, axis=-1) @ vals
        return o
    _patch("tree_attention", tree_attention)


def gqa_modulo():
    def tree_attention(q, k, v, Kp, Vp, visible):
        T, Hq, dh = q.shape
        Hkv = k.shape[1]
        o = np.zeros((T, Hq, dh))
        for hq in range(Hq):
            hk = hq % Hkv
            keys = np.concatenate([Kp[hk], k[:, hk, :]], axis=0)
            vals = np.concatenate([Vp[hk], v[:, hk, :]], axis=0)
            s = np.where(visible, q[:, hq, :] @ keys.T / np.sqrt(dh), -np.inf)
            o[:, hq, :] = om.softmax(s, axis=-1) @ vals
        return o
    _patch("tree_attention", tree_attention)


def no_ancestor_mask():
    _patch("ancestor_matrix", lambda parents: np.tril(np.ones((len(parents), len(parents)), dtype=bool)))


def position_by_node_id():
    from workloads import gen
    gen.Tree.depths = lambda self: np.arange(self.n, dtype=np.int32)


def drop_attention_residual():
    orig = ov.tree_attention

    def verify_tree(ow, prefix_kv, tree, prefix_len):
        m = ow.shape
        T, P = tree.n, prefix_len
        pos = P + tree.depths()
        visible = np.concatenate([np.ones((T, P), dtype=bool), ov.ancestor_matrix(tree.parents)], axis=1)
        x = ow.embed(tree.tokens)
        ks, vs = [], []
        for l in range(m.n_layers):
            L = ow.layer(l)
            q, k, v = om.split_qkv(om.rmsnorm(x, L["attn_norm"], m.rms_eps), L["w_qkv"], m)
            q, k = om.rope(q, pos[:, None], m.rope_base), om.rope(k, pos[:, None], m.rope_base)
            ks.append(k)
            vs.append(v)
            Kp, Vp = prefix_kv(l)
            x = orig(q, k, v, Kp, Vp, visible).reshape(T, -1) @ L["w_o"].T
            x = x + om.mlp(om.rmsnorm(x, L["mlp_norm"], m.rms_eps), L, m)[0]
        logits = om.rmsnorm(x, ow.final_norm, m.rms_eps) @ ow.lm_head().T
        return ov.VerifyResult(logits, x, ks, vs, None)
    ov.verify_tree = verify_tree
    import oracle
    oracle.verify_tree = verify_tree


def swiglu_swapped():
    def swiglu(h, w_gate_up, w_down):
        f = w_down.shape[1]
        return (om.silu(h @ w_gate_up[f:].T) * (h @ w_gate_up[:f].T)) @ w_down.T
    _patch("swiglu", swiglu)


def moe_unnormalised():
    def moe(h, L, top_k):
        logits = h @ L["w_router"].T
        p = om.softmax(logits, axis=-1)
        out = np.zeros_like(h)
        for r in range(h.shape[0]):
            for e in np.argsort(-p[r], kind="stable")[:top_k]:
                out[r] += p[r, e] * om.swiglu(h[r:r + 1], L["w_gate_up"][e], L["w_down"][e])[0]
        return out, logits
    _patch("moe", moe)


def qkv_kv_swapped():
    def split_qkv(h, w_qkv, m):
        Hq, Hkv, dh = m.n_q_heads, m.n_kv_heads, m.head_dim
        y = h @ w_qkv.T
        q = y[:, : Hq * dh].reshape(-1, Hq, dh)
        v = y[:, Hq * dh: (Hq + Hkv) * dh].reshape(-1, Hkv, dh)
        k = y[:, (Hq + Hkv) * dh:].reshape(-1, Hkv, dh)
        return q, k, v
    _patch("split_qkv", split_qkv)


def accept_no_bonus():
    orig = oa.accept_dfs

    def accept_dfs(tree, pred):
        r = orig(tree, pred)
        return oa.AcceptResult(r.length, r.tokens[:-1], r.path)
    _patch("accept_dfs", accept_dfs)
    import oracle
    oracle.accept_dfs = accept_dfs


def accept_first_child_only():
    def accept_dfs(tree, pred):
        node, path = 0, []
        while True:
            kids = [c for c in range(1, tree.n) if tree.parents[c] == node]
            if not kids or int(tree.tokens[kids[0]]) != int(pred[node]):
                break
            node = kids[0]
            path.append(node)
        return oa.AcceptResult(len(path), [int(tree.tokens[i]) for i in path] + [int(pred[node])], path)
    _patch("accept_dfs", accept_dfs)
    import oracle
    oracle.accept_dfs = accept_dfs


def argmax_last_on_ties():
    def argmax_first(logits):
        rev = np.flip(logits, axis=-1)
        return logits.shape[-1] - 1 - np.argmax(rev, axis=-1)
    _patch("argmax_first", argmax_first)
    import oracle
    oracle.argmax_first = argmax_first


def latency_missing_depth():
    import oracle.latency as ol
    ol.speedup_ratio = lambda t, t_bar, d, tau: t / (t + t_bar) * tau
    import oracle
    oracle.speedup_ratio = ol.speedup_ratio


def _sampled_with(kept_in_q=False, unnormalised=False, inverted=False):
    """accept_sampled with one mistake in the rejection step."""
    def accept_sampled(tree, logits, q_draft, u_accept, u_final, temperature):
        tokens, parents = np.asarray(tree.tokens), np.asarray(tree.parents)
        node, path = 0, []
        while True:
            p = osm.softmax_t(logits[node], temperature)
            q = np.asarray(q_draft[node], dtype=np.float64) / np.sum(q_draft[node])
            nxt = None
            for c in [c for c in range(1, len(tokens)) if int(parents[c]) == node]:
                t = int(tokens[c])
                a = min(1.0, q[t] / p[t]) if inverted else min(1.0, p[t] / q[t])
                if float(u_accept[c]) < a:
                    nxt = c
                    break
                r = np.maximum(p - q, 0.0)
                p = r if unnormalised else r / np.sum(r)
                if not kept_in_q:
                    q = q.copy()
                    q[t] = 0.0
                    q = q / np.sum(q)
            if nxt is None:
                emitted = osm.draw(p, u_final[node])
                break
            path.append(nxt)
            node = nxt
        return oa.AcceptResult(len(path), [int(tokens[c]) for c in path] + [emitted], path)
    return accept_sampled


def _patch_sampled(fn):
    _patch("accept_sampled", fn)
    import oracle
    oracle.accept_sampled = fn


def sampling_rejected_token_kept_in_q():
    _patch_sampled(_sampled_with(kept_in_q=True))


def sampling_residual_unnormalised():
    _patch_sampled(_sampled_with(unnormalised=True))


def sampling_ratio_inverted():
    _patch_sampled(_sampled_with(inverted=True))


def _point_mass_with(kept=False, unnormalised=False):
    """accept_sampled whose deterministic-draft (q_draft None) rule has one
    mistake; drawn drafts keep the oracle's own rule."""
    orig = osm.accept_sampled

    def accept_sampled(tree, logits, q_draft, u_accept, u_final, temperature, trace=None):
        if q_draft is not None:
            return orig(tree, logits, q_draft, u_accept, u_final, temperature, trace)
        tokens, parents = np.asarray(tree.tokens), np.asarray(tree.parents)
        node, path = 0, []
        while True:
            p0 = osm.softmax_t(logits[node], temperature)
            p = p0.copy()
            nxt = None
            for c in [c for c in range(1, len(tokens)) if int(parents[c]) == node]:
                t = int(tokens[c])
                a = (p0[t] if p[t] > 0 else 0.0) if unnormalised else p[t]
                if float(u_accept[c]) < a:
                    nxt = c
                    break
                if not kept:
                    p = p.copy()
                    p[t] = 0.0
                    p = p / np.sum(p)
            if nxt is None:
                emitted = osm.draw(p, u_final[node])
                break
            path.append(nxt)
            node = nxt
        return oa.AcceptResult(len(path), [int(tokens[c]) for c in path] + [emitted], path)
    return accept_sampled


def sampling_point_mass_rejected_token_kept():
    _patch_sampled(_point_mass_with(kept=True))


def sampling_point_mass_residual_unnormalised():
    _patch_sampled(_point_mass_with(unnormalised=True))


def sampling_temperature_ignored():
    def softmax_t(logits, temperature):
        z = np.asarray(logits, dtype=np.float64)
        e = np.exp(z - np.max(z))
        return e / np.sum(e)
    _patch("softmax_t", softmax_t)
    import oracle
    oracle.softmax_t = softmax_t


def _patch_both(name, fn):
    _patch(name, fn)
    import oracle
    setattr(oracle, name, fn)


def draft_tgf_no_residual():
    orig = odr.tgf

    def tgf(dow, F, e):
        h, o = orig(dow, F, e)
        return h, o - h
    _patch_both("tgf", tgf)


def draft_layernorm_no_centring():
    def layernorm(x, g, b, eps):
        return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + eps) * g + b
    _patch_both("layernorm", layernorm)


def draft_heads_swapped():
    orig = odr.draft_forward

    def draft_forward(dow, tree, feats_in, prefix_kv, prefix_len):
        r = orig(dow, tree, feats_in, prefix_kv, prefix_len)
        m = dow.shape.target
        logits = om.rmsnorm(r.regress, dow.target.final_norm, m.rms_eps) @ dow.target.lm_head().T
        return odr.DraftResult(logits, r.regress, r.predict, r.h, r.o, r.y)
    _patch_both("draft_forward", draft_forward)


def draft_topk_probabilities():
    orig = odr.topk_logprobs

    def topk_logprobs(logits, k):
        tok, lp = orig(logits, k)
        return tok, np.exp(lp)
    _patch_both("topk_logprobs", topk_logprobs)


def draft_frontier_by_local_probability():
    """The next frontier ranked by each candidate's own log-probability
    instead of the cumulative score of its path."""
    def expand_tree(root_token, root_feature, step, k, depth, n_total, tree_cls):
        p_tok, p_par, p_cand, p_score = [int(root_token)], [-1], [-1], [0.0]
        feats = [np.asarray(root_feature, dtype=np.float64)]
        cands, local = [], []
        frontier, passes = [0], []
        for t in range(depth):
            ptree = tree_cls(np.array(p_tok, dtype=np.int32), np.array(p_par, dtype=np.int32))
            passes.append(ptree)
            tok, logp, regress = step(ptree, np.stack(feats))
            new = []
            for r in frontier:
                for j in range(k):
                    cands.append((t + 1, r, int(tok[r, j]), p_score[r] + float(logp[r, j])))
                    local.append(float(logp[r, j]))
                    new.append(len(cands) - 1)
            if t + 1 == depth:
                break
            best = sorted(new, key=lambda c: (-local[c], c))[:k]
            frontier = []
            for c in best:
                _, r, token, score = cands[c]
                p_tok.append(token)
                p_par.append(r)
                p_cand.append(c)
                p_score.append(score)
                feats.append(np.asarray(regress[r], dtype=np.float64))
                frontier.append(len(p_tok) - 1)
        chosen = sorted(range(len(cands)), key=lambda c: (-cands[c][3], c))[:n_total]
        rank = {c: i for i, c in enumerate(chosen)}
        order = sorted(chosen, key=lambda c: (cands[c][0], rank[c]))
        index = {c: i + 1 for i, c in enumerate(order)}
        tokens = [int(root_token)] + [cands[c][2] for c in order]
        parents = [-1] + [0 if p_cand[cands[c][1]] < 0 else index.get(p_cand[cands[c][1]], 0) for c in order]
        scores = np.array([0.0] + [cands[c][3] for c in order])
        return odr.Expansion(tree_cls(np.array(tokens, dtype=np.int32), np.array(parents, dtype=np.int32)),
                             scores, passes, np.array([c[3] for c in cands]))
    _patch_both("expand_tree", expand_tree)


MUTATIONS = {f.__name__: f for f in [
    rope_sign, rope_interleaved, rope_freq_exponent, rmsnorm_eps_outside, attention_unscaled,
    gqa_modulo, no_ancestor_mask, position_by_node_id, drop_attention_residual, swiglu_swapped,
    moe_unnormalised, qkv_kv_swapped, accept_no_bonus, accept_first_child_only,
    argmax_last_on_ties, latency_missing_depth, sampling_rejected_token_kept_in_q,
    sampling_residual_unnormalised, sampling_ratio_inverted, sampling_temperature_ignored,
    sampling_point_mass_rejected_token_kept, sampling_point_mass_residual_unnormalised,
    draft_tgf_no_residual, draft_layernorm_no_centring, draft_heads_swapped, draft_topk_probabilities,
    draft_frontier_by_local_probability,
]}


def apply(name: str) -> None:
    MUTATIONS[name]()
