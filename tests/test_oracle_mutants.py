"""The oracle's pins must catch plausible mistakes.

Each case plants one mistake in a copy of the oracle's C source (on the CPU),
builds it, and runs the pin checks of ``test_oracle_pins.py`` that cover that
part of the oracle: at least one of them must fail.  A mutant that every pin
accepts would mean the pins leave that part of the definition unchecked.
"""
import os

import pytest

import oracle
from oracle import build as obuild

import test_oracle_pins as pins

BF16 = [pins.check_bf16_rne, pins.check_adam_step1_closed_form, pins.check_dequant_vs_library]
ADAM = [pins.check_adam_step1_closed_form, pins.check_adam_vs_torch,
        pins.check_adam_multistep_vs_torch, pins.check_adam_zero_betas_closed_form]
QUANT = [pins.check_quant_integer_blocks, pins.check_quant_ties_to_even,
         pins.check_quant_nearest_code, pins.check_quant_symmetry_and_scaling,
         pins.check_quant_special_blocks, pins.check_quant_block_boundaries,
         pins.check_round_trip]
GATHER = [pins.check_dequant_vs_library, pins.check_gather_markers,
          pins.check_gather_is_concatenation, pins.check_round_trip]

I4 = [pins.check_i4_packing, pins.check_i4_integer_blocks, pins.check_i4_ties_and_specials,
      pins.check_i4_nearest_code, pins.check_i4_dequant_reduce]

# (name, text in the committed source, planted replacement, checks that must catch it)
MUTANTS = [
    ("bf16-truncates", "        round_up = 1;\n    else if", "        round_up = 0;\n    else if", BF16),
    ("bf16-ties-away", "round_up = (int)(kept & 1u);", "round_up = 1;", BF16),
    ("bf16-ties-down", "round_up = (int)(kept & 1u);", "round_up = 0;", BF16),
    ("bf16-nan-keeps-sign", "return 0x7FC0u;", "return (uint16_t)((bits >> 16) | 0x40u);", BF16),
    ("adam-no-weight-decay", "theta = theta - lr * wd * theta;", "theta = theta - 0.0 * wd * theta;", ADAM),
    ("adam-l2-and-adamw-swapped", "if (adamw)\n", "if (!adamw)\n", ADAM),
    ("adam-eps-inside-sqrt", "(sqrt(vhat) + eps)", "sqrt(vhat + eps)", ADAM),
    ("adam-no-bias-correction-1", "mom1 / bc1", "mom1", ADAM),
    ("adam-no-bias-correction-2", "mom2 / bc2", "mom2", ADAM),
    ("adam-betas-swapped", "b2 * mom2 + (1.0 - b2)", "b1 * mom2 + (1.0 - b1)", ADAM),
    ("adam-update-sign", "theta = theta - lr * mhat", "theta = theta + lr * mhat", ADAM),
    ("adam-decay-after-update", "theta = theta - lr * wd * theta; /* decoupled decay on the old weight */",
     "(void)0;", ADAM),
    ("adam-step-off-by-one", "pow(b1, (double)step)", "pow(b1, (double)(step + 1))", ADAM),
    ("quant-floor", "rintf(y)", "truncf(y)", QUANT),
    ("quant-half-away", "rintf(y)", "roundf(y)", QUANT),
    ("quant-scale-128", "scales[k] = a / 127.0f;", "scales[k] = a / 128.0f;", QUANT),
    ("quant-inverse-128", "127.0f / (a * pre)", "128.0f / (a * pre)", QUANT),
    ("quant-no-prescale", "pre = 0x1p64f;", "pre = 1.0f;", QUANT),
    ("quant-absmax-skips-first", "for (size_t i = lo; i < hi; i++) {\n            const float xi",
     "for (size_t i = lo + 1; i < hi; i++) {\n            const float xi", QUANT),
    ("quant-nonfinite-ignored", "nonfinite = 1;", "nonfinite = 0;", QUANT),
    ("quant-zero-block-unit-scale", "scales[k] = 0.0f;", "scales[k] = 1.0f;", QUANT),
    ("dequant-block-index", "* scales[i / block];", "* scales[i / block / 2];", GATHER),
    ("gather-block-index", "shard_scales[j][i / block]", "shard_scales[j][i / block / 2]", GATHER),
    ("gather-reversed-shards", "(size_t)j * shard_elems + i", "(size_t)(num_shards - 1 - j) * shard_elems + i",
     GATHER),
    ("i4-nibbles-swapped", "codes[i / 2] |= nib;\n            else", "codes[i / 2] |= (uint8_t)(nib << 4);\n            else", I4),
    ("i4-floor", "float q = rintf((x[i] * pre) * inv);", "float q = floorf((x[i] * pre) * inv);", I4),
    ("i4-scale-8", "scales[k] = a / 7.0f;", "scales[k] = a / 8.0f;", I4),
    ("i4-sign-lost", "return nib >= 8 ? nib - 16 : nib;", "return nib;", I4),
    ("i4-mul-then-add", "acc = fmaf((float)orc_i4_code(src_codes[q], i), src_scales[q][i / block], acc);",
     "acc = (float)orc_i4_code(src_codes[q], i) * src_scales[q][i / block] + acc;", I4),
    ("i4-no-output-scale", "out[i] = acc * scale_out;", "out[i] = acc;", I4),
    ("i4-nonfinite-ignored", "if (!isfinite(x[i]))\n                nonfinite = 1;",
     "if (!isfinite(x[i]))\n                nonfinite = 0;", I4),
    ("refresh-drops-last", "for (size_t i = 0; i < count; i++)", "for (size_t i = 0; i + 1 < count; i++)",
     [pins.check_refresh]),
]


def test_mutant_replacements_apply():
    src = open(obuild.SRC).read()
    for name, old, new, _ in MUTANTS:
        assert src.count(old) >= 1, name


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda m: m[0])
def test_pins_catch_mutant(mutant, tmp_path):
    name, old, new, checks = mutant
    src = open(obuild.SRC).read()
    assert old in src
    mut_src = tmp_path / "mutant.c"
    mut_src.write_text(src.replace(old, new, 1))
    lib = obuild.build_oracle(extra_flags=["-Wno-error"], out=str(tmp_path / ("lib_%s.so" % name)),
                             src=str(mut_src))
    orc = oracle.Oracle(lib)
    caught = []
    for check in checks:
        try:
            check(orc)
        except AssertionError:
            caught.append(check.__name__)
    assert caught, "no pin caught mutant %s" % name


def test_unmutated_build_passes_all_checks(tmp_path):
    lib = obuild.build_oracle(out=str(tmp_path / "lib_clean.so"))
    orc = oracle.Oracle(lib)
    for check in sorted(set(BF16 + ADAM + QUANT + GATHER + I4), key=lambda c: c.__name__):
        check(orc)
    assert os.path.exists(lib)
