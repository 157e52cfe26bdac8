"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in an oracle function, on the CPU, by replacing
the function for the duration of the case: a mask that keeps one bit too
many or masks the magnitude, a product that skips the mask, drops the bias,
squares a scale or pairs a row with the wrong channel, a stage map off by
one, an activation quantiser that rounds ties away from zero or flips the
zero point, a weight quantiser without the 2^n / (2^n - 1) factor, an
asymmetric layer that ignores its zero point, a convolution with flipped
taps, a bf16 conversion that truncates, a low-rank branch on unrounded
inputs or with its rank components out of order, bit planes stored least
significant first, packed weights with their bytes reversed, channel sums
of the unmasked weights.  It then runs the pins written for
that function and asserts that at least one of them fails.  A pin set that
let such a mistake through would not pin the oracle."""
import numpy as np
import pytest

import oracle
import test_oracle_pins as pins

REAL = {name: getattr(oracle, name) for name in
        ("mask", "masked_linear", "stage_of_step", "act_quant", "weight_quant",
         "masked_linear_asym", "conv3x3", "bf16_round", "lowrank", "pack_planes",
         "pack_weights", "weight_colsums")}


def failures(checks):
    """How many of the (pin, args) checks fail."""
    n = 0
    for fn, args in checks:
        try:
            fn(*args)
        except (AssertionError, ValueError, IndexError):
            n += 1
    return n


# ------------------------------------------------------------------ mutants

def _mask_extra_bit(W, b):
    return REAL["mask"](W, min(b + 1, 8))


def _mask_magnitude(W, b):
    """Sign-magnitude masking instead of dropping two's-complement bits."""
    REAL["mask"](W, b)                      # same argument checks
    k = 8 - b
    w = np.asarray(W).astype(np.int64)
    return (np.sign(w) * ((np.abs(w) >> k) << k)).clip(-128, 127).astype(np.int8)


def _mask_round(W, b):
    """Rounds to the nearest multiple of 2^k instead of flooring."""
    REAL["mask"](W, b)
    k = 8 - b
    w = np.asarray(W).astype(np.int64)
    half = (1 << k) >> 1
    return (((w + half) >> k) << k).clip(-128, 127).astype(np.int8)


def _linear_no_mask(X, W, sx, sw, b, bias=None):
    return REAL["masked_linear"](X, W, sx, sw, 8, bias)


def _linear_no_bias(X, W, sx, sw, b, bias=None):
    return REAL["masked_linear"](X, W, sx, sw, b, None)


def _linear_scale_squared(X, W, sx, sw, b, bias=None):
    return REAL["masked_linear"](X, W, sx * sx, sw, b, bias)


def _linear_channel_shift(X, W, sx, sw, b, bias=None):
    return REAL["masked_linear"](X, np.roll(np.asarray(W), 1, axis=0), sx, sw, b, bias)


def _linear_drop_last_k(X, W, sx, sw, b, bias=None):
    X, W = np.asarray(X), np.asarray(W)
    if X.shape[1] > 1:
        X, W = X[:, :-1], W[:, :-1]
    return REAL["masked_linear"](X, W, sx, sw, b, bias)


def _stage_off_by_one(t, S, T):
    return REAL["stage_of_step"](min(t + 1, T - 1), S, T)


def _stage_reversed(t, S, T):
    return S - 1 - REAL["stage_of_step"](t, S, T)


def _act_ties_away(x):
    a, z, q = REAL["act_quant"](x)
    x = np.asarray(x, np.float32)
    q2 = np.clip(np.floor(x / np.float32(a) + np.float32(z) + np.float32(0.5)), 0, 255)
    return a, z, q2.astype(q.dtype)


def _act_zero_point_negated(x):
    a, z, q = REAL["act_quant"](x)
    return a, -z, q


def _act_scale_over_256(x):
    a, z, q = REAL["act_quant"](x)
    return a * 255.0 / 256.0, z, q


def _wq_no_grid_factor(W, nbits=8):
    Q, alpha, z, sw = REAL["weight_quant"](W, nbits)
    return Q, alpha, z, np.asarray(alpha, np.float32).copy()


def _wq_round(W, nbits=8):
    Q, alpha, z, sw = REAL["weight_quant"](W, nbits)
    W = np.asarray(W, np.float32)
    q = np.rint(W / np.asarray(alpha, np.float32)[:, None] + np.asarray(z, np.float32)[:, None])
    return np.clip(q, 0, 2 ** nbits - 1).astype(Q.dtype), alpha, z, sw


def _asym_ignores_zero_point(Q, W, alpha, z, sw, b, bias=None):
    return REAL["masked_linear_asym"](Q, W, alpha, 128.0, sw, b, bias)


def _asym_unsigned_acc(Q, W, alpha, z, sw, b, bias=None):
    acc, y = REAL["masked_linear_asym"](Q, W, alpha, z, sw, b, bias)
    Wb = REAL["mask"](np.asarray(W), b).astype(np.int64)
    return np.asarray(Q).astype(np.int64) @ Wb.T, y


def _conv_flipped_taps(X, Wt, sx, sw, b, bias=None):
    return REAL["conv3x3"](X, np.ascontiguousarray(np.asarray(Wt)[:, ::-1, ::-1, :]), sx, sw, b,
                           bias)


def _bf16_truncate(x):
    return (np.asarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16)


def _lowrank_unrounded_input(x, down, up):
    """The fp32 input used as it is instead of rounded to bfloat16."""
    D, U = oracle.bf16_value(down), oracle.bf16_value(up)
    T = np.asarray(x, np.float32).astype(np.float64) @ D.T
    return T, T @ U.T


def _lowrank_rank_order_reversed(x, down, up):
    T, lr = REAL["lowrank"](x, down, up)
    U = oracle.bf16_value(up)
    return T, T @ U[:, ::-1].T


def _planes_lsb_first(W):
    return np.ascontiguousarray(REAL["pack_planes"](W)[:, ::-1])


def _packed_chunk_bytes_reversed(W):
    P = np.asarray(REAL["pack_weights"](W))
    return np.ascontiguousarray(P.reshape(-1, 16)[:, ::-1]).reshape(P.shape)


def _colsums_unmasked(W):
    cs = REAL["weight_colsums"](W)
    return np.repeat(cs[7:8], cs.shape[0], axis=0)


# --------------------------------------------------------------- pin groups

MASK_PINS = ([(pins.test_mask_exhaustive_vs_unsigned_codes, (b,)) for b in range(1, 9)] +
             [(pins.test_mask_exhaustive_vs_bitwise_and, (b,)) for b in range(1, 9)] +
             [(pins.test_mask_worked_values, ()), (pins.test_mask_properties, ())])

LINEAR_PINS = ([(pins.test_b8_equals_numpy_int64_matmul, s)
                for s in [(1, 1, 1), (3, 5, 7), (17, 33, 64), (40, 24, 1153)]] +
               [(pins.test_masked_product_linearity, (b,)) for b in range(1, 9)] +
               [(pins.test_brute_force_agreement, (seed,)) for seed in range(3)] +
               [(pins.test_special_cases, ()), (pins.test_dequant_exact_rational, ()),
                (pins.test_dequant_power_of_two_scales_exact, ())])

STAGE_PINS = [(pins.test_stage_map_golden, ())]

ACT_PINS = ([(pins.test_act_quant_exact_grid_and_ties, ()),
             (pins.test_act_quant_constant_tensor, ())] +
            [(pins.test_act_quant_properties, (seed,)) for seed in range(4)])

WQ_PINS = ([(pins.test_weight_quant_exact_grid_and_clamp, ()),
            (pins.test_weight_quant_truncquant_prefix, ()),
            (pins.test_weight_quant_constant_row, ())] +
           [(pins.test_weight_quant_properties, (seed,)) for seed in (1, 2, 3)])

ASYM_PINS = ([(pins.test_asym_linear_factored_form_and_signed_codes, (b,)) for b in (8, 5, 2)] +
             [(pins.test_asym_linear_reduces_to_symmetric, ())])

CONV_PINS = ([(pins.test_conv_direct_vs_im2col, s)
              for s in [(1, 1, 1, 1), (4, 5, 3, 6), (7, 3, 16, 9)]] +
             [(pins.test_conv_single_tap, ())])

BF16_PINS = ([(pins.test_bf16_round_worked_values, xb) for xb in pins.BF16_WORKED] +
             [(pins.test_bf16_round_matches_torch_rne, ())])

LOWRANK_PINS = [(pins.test_lowrank_exact_rational_tiny, ()), (pins.test_lowrank_merged_weight, ()),
                (pins.test_lowrank_one_hot, ()), (pins.test_lowrank_entries_match_full, ())]

PLANES_PINS = ([(pins.test_planes_bit_position_worked_example, ())] +
               [(pins.test_planes_round_trip, s)
                for s in [(1, 1), (5, 31), (7, 32), (3, 100), (4, 300), (40, 200)]] +
               [(pins.test_bit_plane_identity, (b,)) for b in range(1, 9)])

PACKED_PINS = ([(pins.test_packed_weights_worked_positions, ())] +
               [(pins.test_packed_weights_round_trip, s)
                for s in [(1, 1), (5, 31), (32, 128), (33, 129), (70, 300)]])

COLSUM_PINS = [(pins.test_weight_colsums, ())]

CASES = [
    ("mask", _mask_extra_bit, MASK_PINS),
    ("mask", _mask_magnitude, MASK_PINS),
    ("mask", _mask_round, MASK_PINS),
    ("masked_linear", _linear_no_mask, LINEAR_PINS),
    ("masked_linear", _linear_no_bias, LINEAR_PINS),
    ("masked_linear", _linear_scale_squared, LINEAR_PINS),
    ("masked_linear", _linear_channel_shift, LINEAR_PINS),
    ("masked_linear", _linear_drop_last_k, LINEAR_PINS),
    ("stage_of_step", _stage_off_by_one, STAGE_PINS),
    ("stage_of_step", _stage_reversed, STAGE_PINS),
    ("act_quant", _act_ties_away, ACT_PINS),
    ("act_quant", _act_zero_point_negated, ACT_PINS),
    ("act_quant", _act_scale_over_256, ACT_PINS),
    ("weight_quant", _wq_no_grid_factor, WQ_PINS),
    ("weight_quant", _wq_round, WQ_PINS),
    ("masked_linear_asym", _asym_ignores_zero_point, ASYM_PINS),
    ("masked_linear_asym", _asym_unsigned_acc, ASYM_PINS),
    ("conv3x3", _conv_flipped_taps, CONV_PINS),
    ("bf16_round", _bf16_truncate, BF16_PINS),
    ("lowrank", _lowrank_unrounded_input, LOWRANK_PINS),
    ("lowrank", _lowrank_rank_order_reversed, LOWRANK_PINS),
    ("pack_planes", _planes_lsb_first, PLANES_PINS),
    ("pack_weights", _packed_chunk_bytes_reversed, PACKED_PINS),
    ("weight_colsums", _colsums_unmasked, COLSUM_PINS),
]


def test_pins_pass_on_the_real_oracle():
    """Every pin group passes unmodified (so a failure below is the mutant's)."""
    for group in (MASK_PINS, LINEAR_PINS, STAGE_PINS, ACT_PINS, WQ_PINS, ASYM_PINS, CONV_PINS,
                  BF16_PINS, LOWRANK_PINS, PLANES_PINS, PACKED_PINS, COLSUM_PINS):
        assert failures(group) == 0


@pytest.mark.parametrize("name,mutant,checks", CASES, ids=[c[1].__name__ for c in CASES])
def test_planted_mistake_fails_a_pin(monkeypatch, name, mutant, checks):
    monkeypatch.setattr(oracle, name, mutant)
    assert failures(checks) >= 1, f"no pin of oracle.{name} caught {mutant.__name__}"
