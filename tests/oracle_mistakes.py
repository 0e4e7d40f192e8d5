"""Plausible mistakes planted into the oracle, one at a time, on the CPU.

Each entry names an oracle function and one or more source edits that turn
it into a wrong-but-plausible version (a dropped term, a wrong sign, index,
constant or operand).  ``plant(name)`` compiles the edited function in its
own module's namespace and puts it in place of the original everywhere the
oracle package refers to it.  The pins must catch every one of them:
``tests/test_planted_mistakes.py`` runs the oracle's pin tests once per
mistake (in a child pytest with AVITS_PLANT_MISTAKE set) and requires a
failure each time.
"""
from __future__ import annotations

import importlib
import inspect
import sys
import textwrap

# name -> (module, function, [(original text, planted text), ...])
MISTAKES = {
    # block internals
    "modulation_swapped": ("oracle.block", "_modulate",
                           [("(1.0 + _f64(scale)) + _f64(shift)", "(1.0 + _f64(shift)) + _f64(scale)")]),
    "modulation_without_one": ("oracle.block", "_modulate",
                               [("(1.0 + _f64(scale))", "_f64(scale)")]),
    "rope_sign": ("oracle.block", "apply_rope",
                  [("x0 * c - x1 * s", "x0 * c + x1 * s"), ("x0 * s + x1 * c", "-x0 * s + x1 * c")]),
    "rope_frequency_exponent": ("oracle.block", "rope_angles",
                                [("theta ** (-2.0 * m / n)", "theta ** (-1.0 * m / n)")]),
    "rope_axis_split_order": ("oracle.block", "rope_axes",
                              [("(d // 8, 7 * d // 16, 7 * d // 16)", "(7 * d // 16, 7 * d // 16, d // 8)")]),
    "attention_scale_1_over_d": ("oracle.block", "attention",
                                 [("scale = 1.0 / np.sqrt(d)", "scale = 1.0 / d")]),
    "attention_lse_without_max": ("oracle.block", "attention",
                                  [("m[:, 0] + np.log(l[:, 0])", "np.log(l[:, 0])")]),
    "gelu_constant": ("oracle.block", "gelu_tanh", [("(x + 0.044715 * x", "(x + 0.04715 * x")]),
    "rms_norm_without_gain": ("oracle.block", "rms_norm", [(" * _f64(g)", "")]),
    "layer_norm_without_mean": ("oracle.block", "layer_norm",
                                [("(x - mu) / np.sqrt(var + eps)", "x / np.sqrt(var + eps)")]),
    "double_block_wrong_mlp_gate": ("oracle.block", "double_block",
                                    [("y + mod[5] * (", "y + mod[2] * (")]),
    "double_block_key_from_query_rows": ("oracle.block", "double_block",
                                         [("k = h @ W[D:2 * D].T + b[D:2 * D]", "k = h @ W[:D].T + b[:D]")]),
    "double_block_text_weights_for_images": ("oracle.block", "double_block",
                                             [("(n_txt, S, w_img)):\n        if hi <= lo:\n            continue\n"
                                               "        mod, W, b",
                                               "(n_txt, S, w_txt)):\n        if hi <= lo:\n            continue\n"
                                               "        mod, W, b")]),
    "single_block_without_gate": ("oracle.block", "single_block",
                                  [("x[rows] + mod[2] * y", "x[rows] + y")]),
    "block_qk_unrotated_keys": ("oracle.block", "block_qk",
                                [("return apply_rope(q, ang), apply_rope(k, ang)", "return apply_rope(q, ang), k")]),
    # importance
    "spatial_head_sum": ("oracle.importance", "spatial_importance", [("return acc / H", "return acc")]),
    "spatial_without_lse": ("oracle.importance", "spatial_importance",
                            [("np.exp(p - row_lse[h][:, None])", "np.exp(p)")]),
    "joint_lse_drops_max": ("oracle.importance", "joint_lse",
                            [("m[:, 0] + np.log(np.exp(p - m)", "np.log(np.exp(p - m)")]),
    "text_mass_off_by_one": ("oracle.importance", "text_attention_mass", [("e[:, :L]", "e[:, :L + 1]")]),
    "variance_divisor": ("oracle.importance", "step_variance", [("/ (n_t - 1)", "/ n_t")]),
    "minmax_without_min": ("oracle.importance", "minmax_normalise", [("(hi - lo + eps)", "(hi + eps)")]),
    "fuse_weights_swapped": ("oracle.importance", "joint_score",
                             [("alpha * minmax_normalise(a, eps) + (1.0 - alpha) * minmax_normalise(v, eps)",
                               "alpha * minmax_normalise(v, eps) + (1.0 - alpha) * minmax_normalise(a, eps)")]),
    "mass_score_count_ignored": ("oracle.importance", "score_from_mass",
                                 [("(mass_sum.shape[0] * count)", "mass_sum.shape[0]")]),
    # selection
    "tie_highest_index_wins": ("oracle.selection", "select_topk",
                               [("np.lexsort((idx, key, nan))", "np.lexsort((-idx, key, nan))")]),
    "nan_ranks_as_zero": ("oracle.selection", "select_topk",
                          [("np.lexsort((idx, key, nan))", "np.lexsort((idx, key))")]),
    "perturbation_subtracted": ("oracle.selection", "select_topk_perturbed",
                                [("np.float32) + np.asarray(delta", "np.float32) - np.asarray(delta")]),
    # re-layout
    "canvas_select_inverted": ("oracle.relayout", "gather_upsample",
                               [("np.where(mask[:, None], highres_prev, up)",
                                 "np.where(mask[:, None], up, highres_prev)")]),
    "nearest_transposed_cell": ("oracle.relayout", "upsample_nearest",
                                [("g[r // 2, c // 2]", "g[c // 2 % H_lr, r // 2 % W_lr]")]),
    "bilinear_align_corners": ("oracle.relayout", "upsample_bilinear",
                               [("src = max((o + 0.5) / 2.0 - 0.5, 0.0)", "src = o * (n_in - 1) / max(n_out - 1, 1)")]),
    "positions_row_col_swapped": ("oracle.relayout", "selected_positions",
                                  [("pos[:, 1] = idx // W_hr\n    pos[:, 2] = idx % W_hr",
                                    "pos[:, 2] = idx // W_hr\n    pos[:, 1] = idx % W_hr")]),
    # coordinate-bound noise
    "philox_key_bumped_before_first_round": ("oracle.noise", "philox4x32_10", [("        if r:\n", "        if r >= 0:\n")]),
    "philox_products_swapped": ("oracle.noise", "philox4x32_10",
                                [("hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0", "hi0 ^ x1 ^ k0, lo0, hi1 ^ x3 ^ k1, lo1")]),
    "uniform_without_half": ("oracle.noise", "uniform24", [("+ 0.5) * 2.0 ** -24", ") * 2.0 ** -24")]),
    "box_muller_cos_sin_swapped": ("oracle.noise", "box_muller",
                                   [("out[:, a] = r * np.cos(th)", "out[:, a] = r * np.sin(th)"),
                                    ("out[:, a + 1] = r * np.sin(th)", "out[:, a + 1] = r * np.cos(th)")]),
    "noise_channel_counter_word": ("oracle.noise", "pixel_noise_bits",
                                   [("ctr[:, :, 1] = j[None, :]", "ctr[:, :, 2] = j[None, :]")]),
    "block_noise_plain_mean": ("oracle.noise", "block_noise", [("return acc / 2.0", "return acc / 4.0")]),
    "reinject_weights_swapped": ("oracle.noise", "reinject",
                                 [("(1.0 - float(t)) * np.asarray(x, dtype=np.float64) + float(t) * np.asarray(eps",
                                   "float(t) * np.asarray(x, dtype=np.float64) + (1.0 - float(t)) * np.asarray(eps")]),
    # three-stage sampler
    "clean_estimate_sign_stage2": ("oracle.sampler", "transition12",
                                   [("x0 = euler_update(z, v, -t_s)", "x0 = euler_update(z, v, t_s)")]),
    "clean_estimate_sign_stage3": ("oracle.sampler", "transition23",
                                   [("x0 = euler_update(z_mix, v, -t_s)", "x0 = euler_update(z_mix, v, t_s)")]),
    "collection_starts_early": ("oracle.sampler", "stage1", [("collect = i >= n1", "collect = i >= n1 - 1")]),
    "mass_of_text_rows": ("oracle.sampler", "stage1", [("mass += m[:, L:]", "mass += m[:, :Mp]")]),
    "kept_rows_not_upsampled": ("oracle.sampler", "transition23",
                                [("_, _, full = gather_upsample(state, canvas, None, children, H_lr, W_lr)",
                                  "full = canvas")]),
    # sampler
    "final_layer_without_one": ("oracle.sampler", "final_layer", [("(1.0 + _f64(scale))", "_f64(scale)")]),
    "euler_sign": ("oracle.sampler", "euler_update", [("_f64(z) + float(dt)", "_f64(z) - float(dt)")]),
}


def plant(name: str) -> None:
    """Replace one oracle function by its planted-mistake version."""
    modname, fname, edits = MISTAKES[name]
    importlib.import_module("oracle")
    mod = importlib.import_module(modname)
    orig = getattr(mod, fname)
    src = textwrap.dedent(inspect.getsource(orig))
    for old, new in edits:
        n = src.count(old)
        if n != 1:
            raise RuntimeError(f"planted mistake {name}: {old!r} occurs {n} times in {modname}.{fname}")
        src = src.replace(old, new)
    ns = dict(mod.__dict__)
    exec(compile(src, f"<planted {name}>", "exec"), ns)
    # Rebuilt on the module's own globals, so it sees the module as it is.
    new = type(orig)(ns[fname].__code__, mod.__dict__, fname, orig.__defaults__, orig.__closure__)
    new.__kwdefaults__ = orig.__kwdefaults__
    for m in list(sys.modules.values()):
        mn = getattr(m, "__name__", "") or ""
        if mn == "oracle" or mn.startswith("oracle."):
            for attr, val in list(vars(m).items()):
                if val is orig:
                    setattr(m, attr, new)
