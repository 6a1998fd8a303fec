"""Plant plausible mistakes in the oracle (on the CPU) and show that a pin
catches each one.  Every mutation is a copy of an oracle module with one
function replaced; the real oracle is never modified."""
import copy
import math
import types

import numpy as np
import pytest

import oracle.par as P
import oracle.route as R
import oracle.attn as A
import oracle.coupled as OC
import test_oracle_coupled as TC
import oracle.frame_select as FS
import test_oracle_frame_select as TFS
import oracle.diagnostics as DG
import test_oracle_diagnostics as TDG
import test_oracle_par as TP
import test_oracle_route_attn as TR


def clone(mod, **repl):
    m = types.ModuleType(mod.__name__ + "_mut")
    m.__dict__.update(copy.copy(mod.__dict__))
    m.__dict__.update(repl)
    # rebind module-level functions so internal calls see the replacements
    for name, obj in list(m.__dict__.items()):
        if isinstance(obj, types.FunctionType) and obj.__module__ == mod.__name__ and name not in repl:
            m.__dict__[name] = types.FunctionType(obj.__code__, m.__dict__, name,
                                                  obj.__defaults__, obj.__closure__)
    return m


def _cross_no_conj(Fa, Fb):
    return (Fb * Fa).sum(-1), (np.abs(Fb) * np.abs(Fa)).sum(-1)


def _cross_swapped(Fa, Fb):
    return (Fa * np.conj(Fb)).sum(-1), (np.abs(Fb) * np.abs(Fa)).sum(-1)


def _blend_sign(Fa, Fb, theta, gate, alpha):
    ua = np.exp(-1j * gate * alpha * theta)[..., None]
    ub = np.exp(1j * gate * (1 - alpha) * theta)[..., None]
    return (1 - alpha) * Fa * ua + alpha * Fb * ub


def _blend_alpha_swapped(Fa, Fb, theta, gate, alpha):
    ua = np.exp(1j * gate * alpha * theta)[..., None]
    ub = np.exp(-1j * gate * (1 - alpha) * theta)[..., None]
    return alpha * Fa * ua + (1 - alpha) * Fb * ub


def _blend_drop_gate(Fa, Fb, theta, gate, alpha):
    return P.blend(Fa, Fb, theta, np.ones_like(gate), alpha)


def _dft_sign(n, sign):
    k = np.arange(n)
    return np.exp(-sign * 2j * np.pi * np.outer(k, k) / n)


def _wrap_no_canon(z):
    return math.atan2(z.imag, z.real)


def _bin_tables_kappa1(hp, wp):
    kind, partner, kappa, nu = P.bin_tables(hp, wp)
    return kind, partner, np.ones_like(kappa), nu


def _bin_tables_mirror_swap(hp, wp):
    kind, partner, kappa, nu = P.bin_tables(hp, wp)
    kind = kind.copy()
    rep, mir = kind == P.REP, kind == P.MIRROR
    self_col = np.zeros_like(rep)
    self_col[:, 0] = True
    if wp % 2 == 0:
        self_col[:, wp // 2] = True
    kind[rep & self_col] = P.MIRROR
    kind[mir] = P.REP
    return kind, partner, kappa, nu


def _composition_clip(anchors, n):
    return [(t, a, b, min(max(al, 0.0), 1.0)) for (t, a, b, al) in P.composition(anchors, n)]


def _composition_wrong_pair(anchors, n):
    a = list(anchors)
    out = []
    for (t, pa, pb, al) in P.composition(anchors, n):
        if t > a[-1]:
            pa, pb = a[0], a[1]
            al = (t - pa) / (pb - pa)
        out.append((t, pa, pb, al))
    return out


def _anchor_update_twice(out, resid, anchors, accumulate):
    for a in anchors:
        out[a] = out[a] + 2.0 * resid[a] if accumulate else resid[a]


def _anchor_update_skip_last(out, resid, anchors, accumulate):
    for a in list(anchors)[:-1]:
        out[a] = out[a] + resid[a] if accumulate else resid[a]


def _anchor_update_always_adds(out, resid, anchors, accumulate):
    for a in anchors:
        out[a] = out[a] + resid[a]


PAR_MUTANTS = {
    "cross_no_conj": dict(cross_spectrum=_cross_no_conj),
    "cross_swapped": dict(cross_spectrum=_cross_swapped),
    "blend_sign": dict(blend=_blend_sign),
    "blend_alpha_swapped": dict(blend=_blend_alpha_swapped),
    "blend_drop_gate": dict(blend=_blend_drop_gate),
    "dft_sign": dict(dft_matrix=_dft_sign),
    "wrap_no_canon": dict(wrap_arg=_wrap_no_canon),
    "kappa_all_one": dict(bin_tables=_bin_tables_kappa1),
    "mirror_rep_swapped": dict(bin_tables=_bin_tables_mirror_swap),
    "anchor_update_twice": dict(anchor_update=_anchor_update_twice),
    "anchor_update_skip_last": dict(anchor_update=_anchor_update_skip_last),
    "anchor_update_always_adds": dict(anchor_update=_anchor_update_always_adds),
}


def _any_pin_fails(mod, pins):
    for pin in pins:
        try:
            pin(mod)
        except AssertionError:
            return pin.__name__
    return None


@pytest.mark.parametrize("name", sorted(PAR_MUTANTS))
def test_par_mutation_caught(name):
    mod = clone(P, **PAR_MUTANTS[name])
    caught = _any_pin_fails(mod, TP.PINS)
    assert caught, f"no PAR pin catches mutation {name}"


# Mistakes in App. A.2's reliability rule, planted by editing tile_stats' source.
ETA_MUTANTS = {
    "eta_from_mean_W": ("prm.eta_rel * W.max()", "prm.eta_rel * W.mean()"),
    "eta_max_without_dc": ("prm.eta_rel * W.max()", "prm.eta_rel * W.ravel()[1:].max()"),
    "drop_absZ_leg": ("(W > eta) & (np.abs(Z) > eta)", "(W > eta)"),
    "either_leg": ("(W > eta) & (np.abs(Z) > eta)", "(W > eta) | (np.abs(Z) > eta)"),
    "drop_eta_abs": ("+ prm.eta_abs", "+ 0.0"),
    "omega_plus_drops_nyquist": ("omega_plus[0, 0] = False",
                                 "omega_plus[0, 0] = False; omega_plus[:, 0] &= kind[:, 0] != SELF"),
}


@pytest.mark.parametrize("name", sorted(ETA_MUTANTS))
def test_reliability_mutation_caught(name):
    import inspect
    old, new = ETA_MUTANTS[name]
    text = inspect.getsource(P.tile_stats)
    bad = text.replace(old, new)
    assert bad != text, name
    ns = dict(P.__dict__)
    exec(compile(bad, "<mutant>", "exec"), ns)
    mod = clone(P, tile_stats=ns["tile_stats"])
    caught = _any_pin_fails(mod, TP.PINS)
    assert caught, f"no PAR pin catches mutation {name}"


# Mistakes in eq:gate (tile_stats) and in the per-head routing loop, planted by
# editing the functions' source.
SOURCE_MUTANTS = {
    "gate_tau_linear_in_nu": (P, "tile_stats", "nu ** prm.q", "nu"),
    "route_one_head_for_all": (R, "route", "topk_select(sd[i, h], k_eff)", "topk_select(sd[i, 0], k_eff)"),
    "route_budget_off_by_one": (R, "route", "k_eff = min(int(topk), M)",
                                "k_eff = int(topk) if int(topk) <= M else M - 1"),
    "coupled_pooled_scores_unscaled": (OC, "pooled_stats", "s = scale * (qb @ kb.T)", "s = (qb @ kb.T)"),
    "band_edge_goes_low": (DG, "band_index", 'side="right"', 'side="left"'),
    "progress_frames_shifted": (DG, "phase_progress_frames", "= prog[1:-1]", "= prog[:-2]"),
    "progress_frames_wrong_end": (DG, "phase_progress_frames", "phase_progress(ph, 0, b - a)",
                                  "phase_progress(ph, 0, b - a - 1)"),
    "progress_frames_not_unwrapped": (DG, "phase_progress_frames", "prog = phase_progress(ph, 0, b - a)",
                                      "prog = (ph - ph[0]) / (ph[-1] - ph[0])"),
}


@pytest.mark.parametrize("name", sorted(SOURCE_MUTANTS))
def test_source_mutation_caught(name):
    import inspect
    mod, fn, old, new = SOURCE_MUTANTS[name]
    text = inspect.getsource(getattr(mod, fn))
    bad = text.replace(old, new)
    assert bad != text, name
    ns = dict(mod.__dict__)
    exec(compile(bad, "<mutant>", "exec"), ns)
    mm = clone(mod, **{fn: ns[fn]})
    pins = {P: TP.PINS, R: TR.ROUTE_PINS, OC: TC.PINS, DG: TDG.PINS}[mod]
    assert _any_pin_fails(mm, pins), f"no pin catches mutation {name}"


def test_composition_mutations_caught():
    cases = TP.load_composition_golden()
    for fn in (_composition_clip, _composition_wrong_pair):
        bad = False
        for n, anchors, rows in cases:
            got = fn(anchors, n)
            if [(t, a, b, round(x, 12)) for t, a, b, x in got] != \
                    [(t, a, b, round(x, 12)) for t, a, b, x in rows]:
                bad = True
        assert bad, fn.__name__


def _key_sum_not_mean(q, k_hist):
    return np.asarray(q, np.float64).mean(axis=1), np.asarray(k_hist, np.float64).sum(axis=1)


def _topk_upper_tie(scores_1d, topk):
    s = [float(x) for x in scores_1d]
    order = sorted(range(len(s)), key=lambda m: (-s[m], -m))
    return sorted(order[:min(topk, len(s))])


def _topk_unsorted(scores_1d, topk):
    s = [float(x) for x in scores_1d]
    order = sorted(range(len(s)), key=lambda m: (-s[m], m))
    return order[:min(topk, len(s))]


def _attn_no_scale(Q, K, V, scale):
    return A.softmax_attention(Q, K, V, 1.0)


def _attn_transposed_v(Q, K, V, scale):
    logits = scale * (Q @ K.T)
    p = np.exp(logits - logits.max(1, keepdims=True))
    p /= p.sum(1, keepdims=True)
    out = np.zeros((Q.shape[0], V.shape[1]))
    for r in range(Q.shape[0]):
        out[r] = (p[r][:, None] * V[::-1]).sum(0)
    return out, np.zeros(Q.shape[0])


ROUTE_MUTANTS = {
    "key_sum_not_mean": dict(pooled_means=_key_sum_not_mean),
    "tie_upper_index": dict(topk_select=_topk_upper_tie),
    "unsorted_output": dict(topk_select=_topk_unsorted),
}
ATTN_MUTANTS = {
    "no_scale": dict(softmax_attention=_attn_no_scale),
    "reversed_values": dict(softmax_attention=_attn_transposed_v),
}


@pytest.mark.parametrize("name", sorted(ROUTE_MUTANTS))
def test_route_mutation_caught(name):
    mod = clone(R, **ROUTE_MUTANTS[name])
    assert _any_pin_fails(mod, TR.ROUTE_PINS), name


@pytest.mark.parametrize("name", sorted(ATTN_MUTANTS))
def test_attn_mutation_caught(name):
    mod = clone(A, **ATTN_MUTANTS[name])
    assert _any_pin_fails(mod, TR.ATTN_PINS), name


# ---- reconstruction-coupled routing
def _gains_no_cross(i, x, u, anchors, n_frames, l_anc=1.0, l_rec=1.0):
    x = np.asarray(x, dtype=np.float64)
    u = np.asarray(u, dtype=np.float64)
    an = [int(a) for a in anchors]
    G = l_anc * u[i].copy()
    if i > 0:
        G += l_rec * OC.interval_coeffs(an[i - 1], an[i])[1] * u[i]
    if i < len(an) - 1:
        G += l_rec * OC.interval_coeffs(an[i], an[i + 1])[0] * u[i]
    return G


def _boundary_signed_cross(anchors, n_frames):
    out = OC.boundary_coeffs(anchors, n_frames)
    res = {}
    for q, (a, b, A_, B_, C_) in out.items():
        ts = range(0, a) if q == "L" else range(b + 1, n_frames)
        C2 = sum(((t - a) / (b - a)) * (1 - (t - a) / (b - a)) for t in ts)
        res[q] = (a, b, A_, B_, C2)
    return res


def _omission_stab_numerator(qb, kb, vb, P_, scale, eps=1e-8):
    _, pi, o_bar = OC.pooled_stats(qb, kb, vb, scale)
    vb = np.asarray(vb, dtype=np.float64)
    coef = pi / (1.0 + eps)
    delta = coef[:, :, None] * (o_bar[:, None, :] - vb[None, :, :])
    proj = np.einsum("dk,imk->imd", np.asarray(P_, np.float64), delta)
    return (proj ** 2).sum(axis=2), delta


def _omission_transposed_proj(qb, kb, vb, P_, scale, eps=1e-8):
    u, delta = OC.omission(qb, kb, vb, P_, scale, eps)
    return (delta ** 2).sum(axis=2) * float((np.asarray(P_) ** 2).mean()), delta


def _gains_boundary_swapped(i, x, u, anchors, n_frames, l_anc=1.0, l_rec=1.0):
    G = OC.gains(i, x, u, anchors, n_frames, l_anc, l_rec)
    an = [int(a) for a in anchors]
    row = {a: r for r, a in enumerate(an)}
    for (a, b, A_, B_, C_) in OC.boundary_coeffs(an, n_frames).values():
        if i == row[a]:
            G += l_rec * (B_ - A_) * np.asarray(u, np.float64)[i]
    return G


COUPLED_MUTANTS = {
    "gain_no_cross_term": dict(gains=_gains_no_cross),
    "boundary_signed_cross": dict(boundary_coeffs=_boundary_signed_cross),
    "omission_stabiliser_numerator": dict(omission=_omission_stab_numerator),
    "omission_projection_ignored": dict(omission=_omission_transposed_proj),
    "gain_boundary_A_B_swapped": dict(gains=_gains_boundary_swapped),
}


@pytest.mark.parametrize("name", sorted(COUPLED_MUTANTS))
def test_coupled_mutation_caught(name):
    mod = clone(OC, **COUPLED_MUTANTS[name])
    assert _any_pin_fails(mod, TC.PINS), name


def test_coupled_refine_mutations_caught():
    """Mistakes in Algorithm 1's loop: accepting ties (no strict decrease), a
    forward-only second pass, any positive improvement accepted (no tolerance),
    the tolerance taken as absolute instead of relative to J, and running every
    pass after one that changed nothing."""
    import inspect
    text = inspect.getsource(OC.refine)
    rule = "(g_new - g_old) > tol * max(J, 1e-8)"
    for bad in (text.replace(rule, "(g_new - g_old) >= 0.0"),
                text.replace("if s % 2 == 0 else range(n_a - 1, -1, -1)", ""),
                text.replace(rule, "(g_new - g_old) > 0.0"),
                text.replace(rule, "(g_new - g_old) > tol"),
                text.replace("        if not changed:\n            break\n", "")):
        assert bad != text
        ns = dict(OC.__dict__)
        exec(compile(bad, "<mutant>", "exec"), ns)
        mod = clone(OC, refine=ns["refine"])
        assert _any_pin_fails(mod, TC.PINS)


# ---- control-aware frame selection
F32 = np.float32


def _fs_normalize_no_min(r, eps=1e-8):
    r = np.asarray(r, dtype=F32)
    return (r / (r.max() + F32(eps))).astype(F32)


def _fs_sensitivity_always_half(rs, eps=1e-8):
    got = [r for r in rs if r is not None]
    if not got:
        return None
    acc = np.zeros(len(got[0]), dtype=F32)
    for r in got:
        acc = acc + FS.normalize(r, eps)
    return (acc / F32(2)).astype(F32)


def _fs_ages_no_reset(h, anchors, n_cur):
    h = np.zeros(n_cur, dtype=np.int64) if h is None else np.asarray(h, dtype=np.int64)
    return h + 1


def _fs_debt_floor(h, n_cur, k_f):
    return (np.asarray(h, dtype=F32) / F32(max(n_cur // k_f, 1))).astype(F32)


def _fs_topk_high_index(s, k_f):
    v = [float(x) for x in s]
    order = sorted(range(len(v)), key=lambda i: (-v[i], -i))
    return sorted(order[:k_f])


def _fs_scores_no_lambda(d, debt, lambda_cov=0.5):
    debt = np.asarray(debt, dtype=F32)
    return debt if d is None else (np.asarray(d, dtype=F32) + debt).astype(F32)


FS_MUTANTS = {
    "normalize_no_min": dict(normalize=_fs_normalize_no_min),
    "sensitivity_always_half": dict(sensitivity=_fs_sensitivity_always_half),
    "ages_no_reset": dict(update_ages=_fs_ages_no_reset),
    "debt_floor": dict(coverage_debt=_fs_debt_floor),
    "topk_high_index": dict(topk_frames=_fs_topk_high_index),
    "scores_no_lambda": dict(scores=_fs_scores_no_lambda),
}


@pytest.mark.parametrize("name", sorted(FS_MUTANTS))
def test_frame_select_mutation_caught(name):
    mod = clone(FS, **FS_MUTANTS[name])
    assert _any_pin_fails(mod, TFS.PINS), f"no frame-selection pin catches mutation {name}"


# ---- spectral diagnostics
def _dg_band_no_kappa(ref_t, approx_t, tile_h, tile_w, edges, eps=1e-8):
    ref = np.asarray(ref_t, dtype=np.float64)
    err = ref - np.asarray(approx_t, dtype=np.float64)
    num = np.zeros(len(edges) - 1)
    for (y0, hp, x0, wp) in P.tiles(ref.shape[0], ref.shape[1], tile_h, tile_w):
        F = P.rfft2_ortho(err[y0:y0 + hp, x0:x0 + wp])
        _, _, _, nu = P.bin_tables(hp, wp)
        e = (np.abs(F) ** 2).sum(axis=2)
        for k, v in zip(DG.band_index(nu, edges).ravel(), e.ravel()):
            num[k] += v
    return num / (num.sum() + eps)


def _dg_nrmse_squared(ref_t, approx_t, eps=1e-8):
    ref = np.asarray(ref_t, dtype=np.float64)
    d = ref - np.asarray(approx_t, dtype=np.float64)
    return float((d * d).sum() / ((ref * ref).sum() + eps))


def _dg_unwrap_none(phases):
    return np.asarray(phases, dtype=np.float64).copy()


def _dg_corrections_swapped(ref_t, anchor_a, anchor_b, alpha, tile_h, tile_w):
    rp, rm = DG.oracle_corrections(ref_t, anchor_a, anchor_b, alpha, tile_h, tile_w)
    return rm, rp


def _dg_phase_error_amplitude_weight(ref_t, anchor_a, theta_tiles, alpha, tile_h, tile_w, eps=1e-8):
    ref = np.asarray(ref_t, dtype=np.float64)
    anc = np.asarray(anchor_a, dtype=np.float64)
    num = den = 0.0
    for p, (y0, hp, x0, wp) in enumerate(P.tiles(ref.shape[0], ref.shape[1], tile_h, tile_w)):
        Ft = P.rfft2_ortho(ref[y0:y0 + hp, x0:x0 + wp])
        Fa = P.rfft2_ortho(anc[y0:y0 + hp, x0:x0 + wp])
        _, _, kappa, _ = P.bin_tables(hp, wp)
        w = kappa[:, :, None] * np.abs(Ft)
        w = np.where((np.abs(Ft) > 0) & (np.abs(Fa) > 0), w, 0.0)
        x = np.angle(Ft) - np.angle(Fa) - alpha * np.asarray(theta_tiles[p])[:, :, None]
        num += float((w * np.abs(DG.wrap_pm_pi(x))).sum())
        den += float(w.sum())
    return num / (den + eps)


def _dg_frame_diag(anchor_of_pair=0, flip_alpha=False, approx_from_anchor=False):
    """frame_diagnostics with one assembly mistake planted."""
    def f(ref, approx, anchors, prm, edges, eps=1e-8):
        ref = np.asarray(ref, dtype=np.float64)
        n = ref.shape[0]
        stats = P.par_stats(ref, anchors, prm)
        out = {}
        for (t, a, b, alpha) in P.composition(anchors, n):
            th = [st.theta for (_, _, _, st) in stats[(a, b)]]
            anc = ref[b] if anchor_of_pair else ref[a]
            al = 1.0 - alpha if flip_alpha else alpha
            ap = approx[a] if approx_from_anchor else approx[t]
            rp, rm = DG.oracle_corrections(ref[t], ref[a], ref[b], alpha, prm.tile_h, prm.tile_w)
            out[t] = dict(nrmse=DG.nrmse(ref[t], ap, eps),
                          bands=DG.band_energy(ref[t], ap, prm.tile_h, prm.tile_w, edges, eps),
                          phase_err=DG.phase_error(ref[t], anc, th, al, prm.tile_h, prm.tile_w, eps),
                          r_phase=rp, r_mag=rm)
        return out
    return f


DG_MUTANTS = {
    "frame_diag_phase_from_anchor_b": dict(frame_diagnostics=_dg_frame_diag(anchor_of_pair=1)),
    "frame_diag_alpha_flipped": dict(frame_diagnostics=_dg_frame_diag(flip_alpha=True)),
    "frame_diag_error_of_anchor": dict(frame_diagnostics=_dg_frame_diag(approx_from_anchor=True)),
    "band_no_kappa": dict(band_energy=_dg_band_no_kappa),
    "nrmse_squared": dict(nrmse=_dg_nrmse_squared),
    "no_unwrap": dict(unwrap_track=_dg_unwrap_none),
    "corrections_swapped": dict(oracle_corrections=_dg_corrections_swapped),
    "phase_error_amplitude_weight": dict(phase_error=_dg_phase_error_amplitude_weight),
}


@pytest.mark.parametrize("name", sorted(DG_MUTANTS))
def test_diagnostics_mutation_caught(name):
    mod = clone(DG, **DG_MUTANTS[name])
    assert _any_pin_fails(mod, TDG.PINS), f"no diagnostics pin catches mutation {name}"
