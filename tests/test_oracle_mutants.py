"""Plant plausible mistakes in copies of the oracle and require that the pins
catch every one of them (CPU only).

Each mutant is a textual edit of oracle/oracle.c (a dropped term, a wrong sign
or index, a swapped operand, a misplaced step): (pattern, replacement[, k])
replaces the k-th occurrence (default 0) of the pattern.  The edited copy is
built into a temporary directory; the real oracle is never modified.
"""
import os
import shutil
import tempfile

import pytest

import oracle
from oracle import build as oracle_build
import pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

MUTANTS = {
    "reduce_wrong_peer_index": [("orc_bf16_to_f32(grads[r][i])", "orc_bf16_to_f32(grads[0][i])")],
    "reduce_dropped_scale": [("g[i] = acc * grad_scale;", "g[i] = acc;")],
    "reduce_reverse_order": [("for (int r = 0; r < R; ++r) acc = acc + orc_bf16_to_f32(grads[r][i]);",
                              "for (int r = R - 1; r >= 0; --r) acc = acc + orc_bf16_to_f32(grads[r][i]);")],
    "adamw_dropped_decay": [("float p = master[i] * decay;", "float p = master[i];")],
    "adamw_decay_after_update": [("float p = master[i] * decay;", "float p = master[i];"),
                                 ("p = p - (step_size * (mn / den));",
                                  "p = (p - (step_size * (mn / den))) * decay;")],
    "adamw_m_sign": [("(b1 * m[i]) + (omb1 * gi)", "(b1 * m[i]) - (omb1 * gi)")],
    "adamw_swapped_betas": [("(b2 * v[i]) + (omb2 * (gi * gi))", "(b1 * v[i]) + (omb2 * (gi * gi))")],
    "adamw_v_not_squared": [("(omb2 * (gi * gi))", "(omb2 * gi)")],
    "adamw_eps_inside_sqrt": [("(sqrtf(vn) / bc2_sqrt) + eps", "sqrtf(vn + eps) / bc2_sqrt")],
    "adamw_no_bias_correction1": [("const float step_size = (float)(lr / bc1);",
                                   "const float step_size = (float)lr;")],
    "adamw_no_bias_correction2": [("const float bc2_sqrt = (float)sqrt(bc2);",
                                   "const float bc2_sqrt = 1.0f;")],
    "adamw_bc2_not_rooted": [("const float bc2_sqrt = (float)sqrt(bc2);",
                              "const float bc2_sqrt = (float)bc2;")],
    "adamw_step_off_by_one": [("pow((double)h->beta1, (double)t)", "pow((double)h->beta1, (double)(t + 1))"),
                              ("pow((double)h->beta2, (double)t)", "pow((double)h->beta2, (double)(t + 1))")],
    "adamw_update_sign": [("p = p - (step_size * (mn / den));", "p = p + (step_size * (mn / den));")],
    "adamw_old_m_in_update": [("p = p - (step_size * (mn / den));", "p = p - (step_size * (m[i] / den));")],
    "adamw_decay_ignores_flags": [("(seg_decay == NULL || seg_decay[s]) ? decay_on : 1.0f", "decay_on")],
    "adamw_working_truncated": [("if (working) working[i] = orc_f32_to_bf16(p);",
                                 "if (working) working[i] = (uint16_t)(*(uint32_t*)&p >> 16);")],
    "fedavg_unnormalised": [("out[k] = (float)((double)w[k] / sum);", "out[k] = w[k];")],
    "fedavg_wrong_replica_index": [("(wn[k] * orc_bf16_to_f32(replicas[k][i]))",
                                    "(wn[k] * orc_bf16_to_f32(replicas[0][i]))")],
    "fedavg_master_as_bf16": [("master_out[i] = acc;",
                               "master_out[i] = orc_bf16_to_f32(orc_f32_to_bf16(acc));")],
    "fedavg_reverse_order": [("for (int k = 0; k < G; ++k) acc = acc + (wn[k] * orc_bf16_to_f32(replicas[k][i]));",
                              "for (int k = G - 1; k >= 0; --k) acc = acc + (wn[k] * orc_bf16_to_f32(replicas[k][i]));")],
    "round_stale_own_replica": [("reps[k] = (k == self_group) ? working : replicas[k];",
                                 "reps[k] = (k == self_group) ? replicas[(k + 1) % G] : replicas[k];")],
    "round_same_step_number": [("&ha, step0 + a, g, master", "&ha, step0, g, master")],
    "round_skips_fedavg": [("rc = orc_fedavg(n, G, reps, weights, master, working);", "rc = 0;")],
    "round_reuses_first_grads": [("grads + (size_t)a * (size_t)R", "grads")],
    "sumsq_off_by_one": [("for (int64_t i = seg_off[s]; i < seg_off[s + 1]; ++i) sum +=",
                          "for (int64_t i = seg_off[s] + 1; i < seg_off[s + 1]; ++i) sum +=")],
    "sumsq_not_squared": [("sum += (double)g[i] * (double)g[i];", "sum += (double)g[i];")],
    "bf16_ties_away": [("(lower == 0x8000u && (upper & 1u))", "(lower == 0x8000u)")],
    "bf16_truncate": [("if (lower > 0x8000u || (lower == 0x8000u && (upper & 1u))) upper += 1u;", "")],
    "bf16_nan_not_quiet": [("return (uint16_t)((u >> 16) | 0x0040u);", "return (uint16_t)(u >> 16);")],
    "bf16_decode_shift": [("uint32_t u = (uint32_t)h << 16;", "uint32_t u = (uint32_t)h << 15;")],
    "wire_truncated": [("wire[i] = orc_f32_to_bf16(acc * grad_scale);",
                        "{ float q = acc * grad_scale; uint32_t b; memcpy(&b, &q, 4); wire[i] = (uint16_t)(b >> 16); }")],
    "wire_unscaled": [("wire[i] = orc_f32_to_bf16(acc * grad_scale);", "wire[i] = orc_f32_to_bf16(acc);")],
    "hsdp_skips_tier2": [("    if (H == 1) {\n      rc = orc_shard_reduce(n, R, ga, grad_scale, g);",
                          "    if (1) {\n      rc = orc_shard_reduce(n, R, ga, grad_scale, g);")],
    "hsdp_own_wire_not_used": [("wires[k] = (k == replica) ? wire : replica_wires",
                                "wires[k] = (k == replica) ? replica_wires[(size_t)a * (size_t)H + (size_t)((k + 1) % H)] : replica_wires")],
    "hsdp_unscaled_tier2": [("rc = orc_shard_reduce(n, H, wires, hsdp_scale, g);",
                             "rc = orc_shard_reduce(n, H, wires, 1.0f, g);")],
    "hsdp_member_swapped": [("    if (member) {\n      for (int k = 0; k < G; ++k)",
                             "    if (!member) {\n      for (int k = 0; k < G; ++k)")],
    "bcast_master_through_bf16": [("    master[i] = recv[i];\n    working[i] = orc_f32_to_bf16(recv[i]);",
                                   "    master[i] = orc_bf16_to_f32(orc_f32_to_bf16(recv[i]));\n    working[i] = orc_f32_to_bf16(recv[i]);")],
    "wire_wrong_peer_index": [("orc_bf16_to_f32(grads[r][i])", "orc_bf16_to_f32(grads[0][i])", 1)],
    "hsdp_same_step_number": [("&ha, step0 + a, g, master", "&ha, step0, g, master", 1)],
    "lr_warmup_off_by_one": [("const double s = (double)(t - 1);", "const double s = (double)t;")],
    "lr_min_ignored": [("    f = f * (1.0 - rho) + rho;\n", "")],
    "lr_full_cosine_cycle": [("f = 0.5 * (1.0 + cos(M_PI * q));", "f = 0.5 * (1.0 + cos(2.0 * M_PI * q));")],
    "clip_no_clamp": [("return (float)(c >= 1.0 ? 1.0 : c);", "return (float)c;")],
    "clip_no_eps": [("(sqrt(total_sumsq) + 1e-6)", "sqrt(total_sumsq)")],
    "clip_no_sqrt": [("(sqrt(total_sumsq) + 1e-6)", "(total_sumsq + 1e-6)")],
    "clip_nan_norm_to_one": [("(float)(c >= 1.0 ? 1.0 : c)", "(float)(c < 1.0 ? c : 1.0)")],
    "clip_ignored": [("    if (rc == 0 && max_grad_norm > 0.0f)\n      orc_clip(n, g, max_grad_norm, clip_totals ? clip_totals + a : NULL);\n", "")],
    "clip_before_sumsq": [("    if (rc == 0 && seg_sumsq)\n      rc = orc_seg_sumsq(n_seg, seg_off, g, seg_sumsq + (size_t)a * (size_t)n_seg);\n    if (rc == 0 && max_grad_norm > 0.0f)\n      orc_clip(n, g, max_grad_norm, clip_totals ? clip_totals + a : NULL);",
                           "    if (rc == 0 && max_grad_norm > 0.0f)\n      orc_clip(n, g, max_grad_norm, clip_totals ? clip_totals + a : NULL);\n    if (rc == 0 && seg_sumsq)\n      rc = orc_seg_sumsq(n_seg, seg_off, g, seg_sumsq + (size_t)a * (size_t)n_seg);")],
    "round_ignores_step_lr": [("    if (step_lr) ha.lr = step_lr[a];\n", "")],
    "round_first_step_lr_only": [("if (step_lr) ha.lr = step_lr[a];", "if (step_lr) ha.lr = step_lr[0];")],
    "hsdp_reuses_first_grads": [("grads + (size_t)a * (size_t)R", "grads", 1)],
    "outer_delta_sign": [("const float delta = prev[i] - xbar;", "const float delta = xbar - prev[i];")],
    "outer_no_momentum": [("const float b = (mu * buf[i]) + delta;", "const float b = delta;")],
    "outer_nesterov_uses_old_buf": [("(delta + (mu * b))", "(delta + (mu * buf[i]))")],
    "outer_nesterov_inverted": [("o->nesterov ? (delta + (mu * b)) : b", "o->nesterov ? b : (delta + (mu * b))")],
    "outer_buf_not_stored": [("    buf[i] = b;\n", "")],
    "outer_prev_not_updated": [("    prev[i] = p;\n", "")],
    "outer_lr_ignored": [("const float p = prev[i] - (eta * d);", "const float p = prev[i] - d;")],
    "outer_unnormalised_weights": [("if (orc_norm_weights(G, weights, wn) != 0) {", "if (orc_norm_weights(G, weights, wn) != 0 || (wn[0] = weights[0], 0)) {", 1)],
    "round_outer_skips_outer": [("rc = orc_fedopt(n, G, reps, weights, o, prev, buf, master, working);", "rc = orc_fedavg(n, G, reps, weights, master, working);")],
    "hsdp_stale_own_replica": [("reps[k] = (k == self_group) ? working : replicas[k];",
                                "reps[k] = (k == self_group) ? replicas[(k + 1) % G] : replicas[k];", 1)],
}


@pytest.fixture(scope="module")
def workdir():
    d = tempfile.mkdtemp(prefix="oracle_mutants_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


def _build_mutant(workdir, name, edits):
    src = open(SRC).read()
    for edit in edits:
        old, new = edit[0], edit[1]
        k = edit[2] if len(edit) > 2 else 0
        pos = -1
        for _ in range(k + 1):
            pos = src.find(old, pos + 1)
            assert pos >= 0, "mutation %s: occurrence %d of %r missing" % (name, k, old)
        src = src[:pos] + new + src[pos + len(old):]
    path = os.path.join(workdir, name + ".c")
    with open(path, "w") as f:
        f.write(src)
    return oracle_build.build(out=os.path.join(workdir, "lib" + name + ".so"), src=path,
                              include_dir=os.path.dirname(SRC))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(workdir, name):
    lib_path = _build_mutant(workdir, name, MUTANTS[name])
    orc = oracle.Oracle(lib_path)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(orc)
        except (AssertionError, ValueError, FloatingPointError) as e:
            caught.append((pin.__name__, str(e)[:120]))
            break
    assert caught, "planted mistake %s passed every pin" % name
