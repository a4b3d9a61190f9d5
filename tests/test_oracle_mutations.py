"""The oracle's pins catch plausible mistakes.

Each case below plants one mistake in the oracle on the CPU: a dropped term,
a wrong sign or index, a transposed operand, an off-by-one.  The pins of
tests/test_oracle_*.py then run against the mutated oracle, and at least one
of them must fail.  A mutant that every pin accepts would be a mistake the
oracle could carry unnoticed.
"""

import math

import numpy as np
import pytest

from oracle import accounting, attention, gradients, hilbert, schedule, tokens
from oracle.schedule import Layout

import test_oracle_accounting as t_acc
import test_oracle_attention as t_att
import test_oracle_attention_rows as t_rows
import test_oracle_general as t_gen
import test_oracle_gradients as t_grad
import test_oracle_hilbert as t_hil
import test_oracle_moved as t_mov
import test_oracle_schedule as t_sch
import test_oracle_tokens as t_tok

# A fast battery of pins over every oracle module.
PINS = [
    lambda: t_hil.test_bijection(3),
    lambda: t_hil.test_consecutive_positions_are_4_neighbours(4),
    lambda: t_hil.test_self_similar_runs_are_aligned_squares(4),
    lambda: t_hil.test_iterative_matches_lsystem(4),
    lambda: t_hil.test_order2_golden_table(),
    lambda: t_hil.test_start_end_corners_and_mirror_symmetry(3),
    lambda: t_sch.test_tiles_partition_the_image(t_sch.LAYOUTS[0], 1),
    lambda: t_sch.test_tiles_partition_the_image(t_sch.LAYOUTS[3], 3),
    lambda: t_sch.test_effective_receptive_field_grows_one_tile_per_layer(64, 16, 4),
    lambda: t_sch.test_tiny_shared_runs_match_hand_derivation(),
    lambda: t_sch.test_flux64_shared_tokens_per_tile(),
    lambda: t_sch.test_mask_properties(t_sch.LAYOUTS[3], 1),
    lambda: t_sch.test_schedule_table_layout(),
    lambda: t_att.test_loop_version_agrees_on_a_real_pattern(),
    lambda: t_att.test_one_tile_is_dense_attention(),
    lambda: t_att.test_slide_equals_roll_then_unshifted_attention(1),
    lambda: t_att.test_global_rows_equal_dense_rows(),
    lambda: t_att.test_lse_is_logsumexp_of_unmasked_logits(),
    lambda: t_att.test_masked_keys_have_no_influence(),
    lambda: t_rows.test_rows_equal_full_oracle_for_every_row_class(t_rows.LAYOUTS[0], 1),
    lambda: t_rows.test_rows_equal_full_oracle_for_every_row_class(t_rows.LAYOUTS[2], 1),
    lambda: t_rows.test_rows_match_the_loop_implementation(),
    lambda: t_tok.test_gather_orders_tokens_along_the_curve(8),
    lambda: t_tok.test_scatter_restores_raster_order(4),
    lambda: t_acc.test_nnz_matches_closed_form(Layout(16, 16, 0, 64, 32, 4, 4), 1, 22_368),
    lambda: t_mov.test_moved_order_is_shared_first_then_hilbert(t_mov.MOVED[1]),
    lambda: t_mov.test_tiles_partition_the_tiled_span(t_mov.MOVED[0], 1),
    lambda: t_mov.test_moved_sequence_equals_raster_construction(t_mov.MOVED[2], 1),
    lambda: t_mov.test_pattern_size_closed_form(t_mov.MOVED[3]),
    lambda: t_gen.test_cells_follow_the_enclosing_turtle_curve(5, 7),
    lambda: t_gen.test_shared_region_is_centred_in_the_grid(),
    lambda: t_gen.test_padded_sequence_equals_raster_construction(t_gen.PADDED[1], 1),
    lambda: t_gen.test_padding_content_does_not_reach_other_rows(t_gen.PADDED[0]),
    lambda: t_grad.test_finite_differences(t_grad.LAYOUTS[0], 1),
    lambda: t_grad.test_matches_torch_autograd(t_grad.LAYOUTS[3], 1),
]


def _xy_transposed(orig):
    def f(order):
        x, y = orig(order)
        return y, x
    return f


def _xy_no_reflection(orig):
    # the digit loop without the reflection of the rx == 1 quadrant
    def f(order):
        side = 1 << order
        d = np.arange(side * side, dtype=np.int64)
        x = np.zeros_like(d)
        y = np.zeros_like(d)
        t, s = d.copy(), 1
        while s < side:
            rx = (t // 2) & 1
            ry = (t ^ rx) & 1
            swap = ry == 0
            x, y = np.where(swap, y, x), np.where(swap, x, y)
            x, y, t, s = x + s * rx, y + s * ry, t // 4, s * 2
        return x, y
    return f


def _labels_off_by_one_tile(orig):
    return lambda layout, layer: (orig(layout, layer) + 1) % layout.n_tiles


def _labels_unslid(orig):
    return lambda layout, layer: orig(layout, 0)


def _shared_shifted(orig):
    def f(layout):
        m = orig(layout).reshape(layout.grid_h, layout.grid_w)
        return np.roll(m, 1, axis=0).reshape(-1)
    return f


def _mask_without_global_keys(orig):
    def f(layout, layer, rows):
        rows = np.asarray(rows, dtype=np.int64)
        is_global, lab = schedule.token_classes(layout, layer)
        m = np.repeat(is_global[rows][:, None], layout.n_tot, axis=1)
        m |= (lab[rows][:, None] == lab[None, :]) & (lab[rows][:, None] >= 0)
        return m
    return f


def _mask_without_global_rows(orig):
    def f(layout, layer, rows):
        rows = np.asarray(rows, dtype=np.int64)
        is_global, lab = schedule.token_classes(layout, layer)
        m = np.repeat(is_global[None, :], len(rows), axis=0)
        m |= (lab[rows][:, None] == lab[None, :]) & (lab[rows][:, None] >= 0)
        m[np.arange(len(rows)), rows] = True
        return m
    return f


def _attention_with(mistake):
    """masked_attention with one planted mistake in its closed form."""
    def f(q, k, v, mask_fn, scale=None, block=1024, empty_rows=False):
        q, k, v = (np.asarray(a, dtype=np.float64) for a in (q, k, v))
        b, h, n, d = q.shape
        scale = 1.0 / math.sqrt(d) if scale is None else scale
        if mistake == "no_scale":
            scale = 1.0
        rows = np.arange(n)
        m = mask_fn(rows)
        s = np.einsum("bhid,bhjd->bhij", q, k) * scale
        if mistake != "no_mask":
            s = np.where(m[None, None], s, -np.inf)
        mx = s.max(axis=-1, keepdims=True)
        p = np.exp(s - mx)
        den = p.sum(axis=-1, keepdims=True)
        vv = k if mistake == "k_for_v" else v
        out = np.einsum("bhij,bhjd->bhid", p, vv)
        if mistake != "no_normalise":
            out = out / den
        lse = (mx + np.log(den))[..., 0]
        if mistake == "lse_without_max":
            lse = np.log(den)[..., 0]
        return out, lse
    return lambda orig: f


def _rows_with(mistake):
    """masked_attention_rows with one planted mistake."""
    def f(q, k, v, rows, mask_rows, scale=None):
        q, k, v = (np.asarray(a, dtype=np.float64) for a in (q, k, v))
        d = q.shape[-1]
        scale = 1.0 / math.sqrt(d) if scale is None else scale
        if mistake == "no_scale":
            scale = 1.0
        rows = np.asarray(rows, dtype=np.int64)
        m = np.asarray(mask_rows)
        if mistake == "mask_row_offset":
            m = np.roll(m, 1, axis=0)
        some = m.any(axis=1)
        s = np.einsum("bhid,bhjd->bhij", q[:, :, rows], k) * scale
        s = np.where(m[None, None], s, -np.inf)
        mx = np.where(some[None, None, :, None], s.max(axis=-1, keepdims=True), 0.0)
        p = np.exp(s - mx)
        den = p.sum(axis=-1, keepdims=True)
        with np.errstate(divide="ignore", invalid="ignore"):
            o = np.einsum("bhij,bhjd->bhid", p, v) / den
            ls = (mx + np.log(den))[..., 0]
        if mistake == "empty_rows_not_zero":
            return o, ls
        return (np.where(some[None, None, :, None], o, 0.0), np.where(some[None, None, :], ls, -np.inf))
    return lambda orig: f


def _permute_through_inverse(orig):
    def f(x, perm):
        inv = np.empty_like(np.asarray(perm, dtype=np.int64))
        inv[np.asarray(perm)] = np.arange(inv.size)
        return orig(x, inv)
    return f


def _nnz_drops_last_block(orig):
    def f(layout, layer, block=2048):
        total = 0
        for r0 in range(0, layout.n_tot - 1, 8):
            rows = np.arange(r0, min(layout.n_tot - 1, r0 + 8))
            total += int(schedule.mask_rows(layout, layer, rows).sum())
        return total
    return f


def _moved_is_the_plain_curve(orig):
    return lambda layout: hilbert.build_perm(layout.grid_h, layout.grid_w)[0]


def _moved_parts_in_raster_order(orig):
    def f(layout):
        sh = schedule.shared_raster(layout)
        return np.concatenate([np.nonzero(sh)[0], np.nonzero(~sh)[0]])
    return f


def _padding_keys_valid(orig):
    return lambda layout: np.ones(layout.n_tot, dtype=bool)


def _padded_grid_transposed(orig):
    return lambda grid_h, grid_w: orig(grid_w, grid_h)


def _region_centred_in_enclosing_grid(orig):
    def f(layout):
        side = layout.side
        r0 = (side - layout.shared_h) // 2
        c0 = (side - layout.shared_w) // 2
        yy, xx = np.divmod(np.arange(layout.grid_h * layout.grid_w), layout.grid_w)
        return ((yy >= r0) & (yy < r0 + layout.shared_h) & (xx >= c0) &
                (xx < c0 + layout.shared_w))
    return f


def _grads_with(mistake):
    """masked_attention_grads with one planted mistake."""
    def f(q, k, v, do, mask_fn, scale=None, block=512):
        q, k, v, do = (np.asarray(a, dtype=np.float64) for a in (q, k, v, do))
        b, h, n, d = q.shape
        scale = 1.0 / math.sqrt(d) if scale is None else scale
        rows = np.arange(n)
        m = mask_fn(rows)
        some = m.any(axis=1)
        s = np.where(m[None, None], np.einsum("bhid,bhjd->bhij", q, k) * scale, -np.inf)
        mx = np.where(some[None, None, :, None], s.max(axis=-1, keepdims=True), 0.0)
        e = np.exp(s - mx)
        den = e.sum(axis=-1, keepdims=True)
        p = e / np.where(den > 0, den, 1.0)
        o = np.einsum("bhij,bhjd->bhid", p, v)
        dlt = np.sum(do * o, axis=-1, keepdims=True)
        dp = np.einsum("bhid,bhjd->bhij", do, v)
        ds = p * dp if mistake == "no_row_term" else p * (dp - dlt)
        dq = (1.0 if mistake == "dq_unscaled" else scale) * np.einsum("bhij,bhjd->bhid", ds, k)
        dk = scale * np.einsum("bhij,bhid->bhjd", ds, k if mistake == "dk_from_k" else q)
        dv = np.einsum("bhij,bhid->bhjd", e if mistake == "dv_unnormalised" else p, do)
        return dq, dk, dv
    return lambda orig: f


MUTANTS = {
    "curve transposed": (hilbert, "xy_iterative", _xy_transposed),
    "curve without reflection": (hilbert, "xy_iterative", _xy_no_reflection),
    "labels off by one tile": (schedule, "labels", _labels_off_by_one_tile),
    "labels ignore the slide": (schedule, "labels", _labels_unslid),
    "shared region one row low": (schedule, "shared_raster", _shared_shifted),
    "mask drops global keys": (schedule, "mask_rows", _mask_without_global_keys),
    "mask drops global rows": (schedule, "mask_rows", _mask_without_global_rows),
    "attention without scale": (attention, "masked_attention", _attention_with("no_scale")),
    "attention ignores mask": (attention, "masked_attention", _attention_with("no_mask")),
    "attention uses K for V": (attention, "masked_attention", _attention_with("k_for_v")),
    "attention not normalised": (attention, "masked_attention", _attention_with("no_normalise")),
    "lse without the max": (attention, "masked_attention", _attention_with("lse_without_max")),
    "sampled rows: mask one row off": (attention, "masked_attention_rows", _rows_with("mask_row_offset")),
    "sampled rows without scale": (attention, "masked_attention_rows", _rows_with("no_scale")),
    "sampled rows: padding rows not empty": (
        attention, "masked_attention_rows", _rows_with("empty_rows_not_zero")),
    "gather through the inverse": (tokens, "permute", _permute_through_inverse),
    "nnz drops the last row": (accounting, "nnz", _nnz_drops_last_block),
    "moved order is the plain curve": (schedule, "moved_perm", _moved_is_the_plain_curve),
    "moved parts in raster order": (schedule, "moved_perm", _moved_parts_in_raster_order),
    "padding attended as keys and queries": (schedule, "token_valid", _padding_keys_valid),
    "general grid transposed": (hilbert, "padded_perm", _padded_grid_transposed),
    "region centred in the enclosing grid": (schedule, "shared_raster", _region_centred_in_enclosing_grid),
    "gradient without the row term": (gradients, "masked_attention_grads", _grads_with("no_row_term")),
    "dQ without the scale": (gradients, "masked_attention_grads", _grads_with("dq_unscaled")),
    "dK from K instead of Q": (gradients, "masked_attention_grads", _grads_with("dk_from_k")),
    "dV from unnormalised P": (gradients, "masked_attention_grads", _grads_with("dv_unnormalised")),
    "moved prefix without the shared tokens": (
        Layout, "prefix", lambda orig: property(lambda self: self.n_txt)),
}


def _failing_pins():
    failed = []
    for i, pin in enumerate(PINS):
        try:
            pin()
        except Exception:  # an assertion, or the oracle rejecting its own output
            failed.append(i)
    return failed


def test_pins_pass_on_the_oracle():
    assert _failing_pins() == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(monkeypatch, name):
    module, attr, make = MUTANTS[name]
    monkeypatch.setattr(module, attr, make(getattr(module, attr)))
    assert _failing_pins(), "no pin catches the mutant '%s'" % name
