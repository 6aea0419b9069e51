"""Plant plausible mistakes in copies of the oracle and check that a pin trips.

Each mutation edits one expression of oracle/lumo_oracle.c (a dropped term, a wrong
sign, a wrong index, a transposed operand, a reversed tap order, a skipped node);
every mutant stays within the bounds of its arrays. The copy is
compiled with gcc into a temporary directory and runs every pin against it.
The real oracle is never modified.
"""
import os
import shutil
import subprocess

import pytest

import oracle
import pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "lumo_oracle.c")

MUTATIONS = {
    "drop_decay": ("for (long e = 0; e < (long)dv * dk; ++e) R[e] *= a;",
                   "for (long e = 0; e < (long)dv * dk; ++e) R[e] *= 1.0;"),
    "drop_beta": ("Rk[j] = b * (vv[j] - s);", "Rk[j] = (vv[j] - s);"),
    "sign_flip": ("Rk[j] = b * (vv[j] - s);", "Rk[j] = b * (vv[j] + s);"),
    "decay_after_dot": ("    /* R' = alpha R */\n    for (long e = 0; e < (long)dv * dk; ++e) R[e] *= a;\n",
                        "    for (long e = 0; e < (long)dv * dk; ++e) R[e] *= 1.0;\n"),
    "transposed_state": ("R[(long)j * d->d_k + i] = (double)state[base + (long)i * d->d_v + j];",
                         "R[(long)j * d->d_k + i] = (double)state[base + (long)j * d->d_k + i];"),
    "head_modulo": ("const int hk = h / (d->h_v / d->h_k);\n    const long kb",
                    "const int hk = h % d->h_k;\n    const long kb"),
    "skip_root_update": ("for (int p = 0; p < len; ++p)\n            gdn_node_update(",
                         "for (int p = 1; p < len; ++p)\n            gdn_node_update("),
    "output_from_parent": ("for (int j = 0; j < dv; ++j)\n        for (int i = 0; i < dk; ++i) R[(long)j * dk + i] += Rk[j] * kv[i];",
                           "for (int j = 0; j < dv; ++j)\n        for (int i = 0; i < dk; ++i) R[(long)j * dk + i] += 0.0 * Rk[j] * kv[i];"),
    "query_head_zero": ("const long qb = (((long)l * d->total_rows + row) * d->h_k + hk) * dk;",
                        "const long qb = (((long)l * d->total_rows + row) * d->h_k + 0) * dk;"),
    "query_row_of_parent": ("gdn_output(d, s.R, l, row[targets[t]], h,",
                            "gdn_output(d, s.R, l, row[s.path[len > 1 ? len - 2 : 0]], h,"),
    "reversed_taps": ("acc += (double)w[((long)l * channels + c) * 4 + t] * xv;",
                      "acc += (double)w[((long)l * channels + c) * 4 + (3 - t)] * xv;"),
    "history_reversed": ("xv = ld_op(hist, (((long)r * n_layers + l) * 3 + pos) * channels + c, op_dtype);",
                         "xv = ld_op(hist, (((long)r * n_layers + l) * 3 + (2 - pos)) * channels + c, op_dtype);"),
    "hist_publish_shift": ("const int pos = L + e;", "const int pos = L + e - 1 < 0 ? 0 : L + e - 1;"),
    "commit_skips_last": ("for (int p = 0; p < path_len[r]; ++p)", "for (int p = 0; p + 1 < path_len[r]; ++p)"),
    "qk_norm_without_eps": ("const double scale = sqrt(ss + d->qk_eps);", "const double scale = sqrt(ss);"),
    "query_not_normalised": ("    qk_prepare(d, qv, dk);\n", ""),
    "raw_gate_without_dt_bias": ("const double x = g_in + (double)d->dt_bias[lh];", "const double x = g_in;"),
    "raw_beta_sign": ("*beta = 1.0 / (1.0 + exp(-b_in));", "*beta = 1.0 / (1.0 + exp(b_in));"),
    "attn_drops_last_context": ("const long c0 = ctx_off[r], nc = ctx_off[r + 1] - ctx_off[r];",
                                "const long c0 = ctx_off[r], nc = ctx_off[r + 1] - ctx_off[r] - (ctx_off[r + 1] > ctx_off[r]);"),
    "attn_kv_head_modulo": ("const int hk = h / grp;", "const int hk = h % h_kv;"),
    "attn_no_scale": ("sc[t] = scale * s;", "sc[t] = s;"),
    "attn_value_of_parent": ("const long vb = t < nc ? ((c0 + t) * h_kv + hk) * d : ((long)rw[path[t - nc]] * h_kv + hk) * d;",
                             "const long vb = t < nc ? ((c0 + t) * h_kv + hk) * d : ((long)rw[path[t - nc > 0 ? t - nc - 1 : 0]] * h_kv + hk) * d;"),
    "attn_excludes_self": ("for (long t = 0; t < nc + len; ++t) {\n                    const void* kk",
                           "for (long t = 0; t < nc + len - (len > 1); ++t) {\n                    const void* kk"),
    "select_tie_reversed": ("return ties == 0 ? ia < ib : ia > ib;", "return ties == 0 ? ia > ib : ia < ib;"),
    "select_nan_lowest": ("if (isnan(a)) return !isnan(b);", "if (isnan(a)) return 0;"),
    "select_spine_last_maximum": ("if (sel_greater(ld_op(logits, base + i, op_dtype), ld_op(logits, base + best, op_dtype))) best = i;",
                                  "if (!sel_greater(ld_op(logits, base + best, op_dtype), ld_op(logits, base + i, op_dtype))) best = i;"),
    "select_repeats_candidates": ("                if (taken) continue;\n", ""),
    "select_spine_skips_index_1": ("for (int i = 1; i < vocab; ++i)\n            if (sel_greater(",
                                   "for (int i = 2; i < vocab; ++i)\n            if (sel_greater("),
    # batch drivers: per-request offsets and per-instance indices
    "verify_all_output_at_node_id": ("double* dst = o_all + (((long)l * d->total_rows + rw[i]) * d->h_v + h) * d->d_v;",
                                     "double* dst = o_all + (((long)l * d->total_rows + i) * d->h_v + h) * d->d_v;"),
    "verify_all_layer_from_head": ("const int l = (int)((inst / d->h_v) % d->n_layers);\n        const int r = (int)(inst / ((long)d->h_v * d->n_layers));\n        const int n = node_off[r + 1] - node_off[r];",
                                   "const int l = (int)(inst % d->n_layers);\n        const int r = (int)(inst / ((long)d->h_v * d->n_layers));\n        const int n = node_off[r + 1] - node_off[r];"),
    "commit_rows_of_request0": ("const int* rw = row + node_off[r];\n        load_state(d, state_in",
                                "const int* rw = row;\n        load_state(d, state_in"),
    "commit_state_of_request0": ("load_state(d, state_in, r, l, h, s.R);", "load_state(d, state_in, 0, l, h, s.R);"),
    "commit_invalid_reports_zero": ("path_len[r] = -1;\n            continue;\n        }\n        int* tmp",
                                    "path_len[r] = 0;\n            continue;\n        }\n        int* tmp"),
    "conv_history_of_request0": ("xv = ld_op(hist, (((long)r * n_layers + l) * 3 + pos) * channels + c, op_dtype);",
                                 "xv = ld_op(hist, (((long)0 * n_layers + l) * 3 + pos) * channels + c, op_dtype);"),
    "conv_rows_of_request0": ("const int* rw = row + node_off[r];\n        int* path = (int*)malloc(sizeof(int) * (size_t)(n > 0 ? n : 1));",
                              "const int* rw = row;\n        int* path = (int*)malloc(sizeof(int) * (size_t)(n > 0 ? n : 1));"),
    "hist_publish_rows_of_request0": ("const int* rw = row + node_off[r];\n        for (int l = 0; l < n_layers; ++l)",
                                      "const int* rw = row;\n        for (int l = 0; l < n_layers; ++l)"),
    "hist_publish_history_of_request0": ("val = ld_op(hist, (((long)r * n_layers + l) * 3 + pos) * channels + c, op_dtype);",
                                         "val = ld_op(hist, (((long)0 * n_layers + l) * 3 + pos) * channels + c, op_dtype);"),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(tmp_path, name):
    old, new = MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique/found"
    mutated = tmp_path / "mut.c"
    mutated.write_text(src.replace(old, new))
    so = tmp_path / "libmut.so"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-o",
                           str(so), str(mutated), "-lm"])
    caught = []
    oracle.use_library(str(so))
    try:
        for pin in pins.ALL_PINS:
            try:
                pin()
            except (AssertionError, ValueError):
                caught.append(pin.__name__)
    finally:
        oracle.use_library(None)
    assert caught, f"no pin detects mutation {name}"
