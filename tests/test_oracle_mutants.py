"""Plant plausible mistakes in copies of the oracle (on the CPU) and check that
the pins catch every one.

Each mutant is a textual edit of oracle/xred_oracle.c compiled into a
temporary directory; the real oracle is untouched.  A mutant "survives" when
every pin passes on it, which would mean the pins cannot tell that mistake
from the correct definition.
"""
import subprocess
import sys
from pathlib import Path

import pytest

ROOT = Path(__file__).resolve().parents[1]
sys.path.insert(0, str(ROOT))

import oracle  # noqa: E402
import pins  # noqa: E402

SRC = (ROOT / "oracle" / "xred_oracle.c").read_text()

# (name, original text, replacement, count of occurrences to replace (0 = all), extra flags)
MUTANTS = [
    ("drop_last_source", "for (int p = 1; p < nsrc; ++p)", "for (int p = 1; p < nsrc - 1; ++p)", 0, ()),
    ("skip_first_source", "for (int p = 1; p < nsrc; ++p)\n            acc = op_float",
     "for (int p = 2; p < nsrc; ++p)\n            acc = op_float", 1, ()),
    ("init_from_zero",
     "float acc = up_float(srcs[0], off + i, dtype);\n        for (int p = 1;",
     "float acc = 0.0f;\n        for (int p = 0;", 1, ()),
    ("bf16_ties_away", "(dropped == 0x8000u && (kept & 1u))", "(dropped == 0x8000u)", 1, ()),
    ("bf16_truncate", "kept += 1u;", "kept += 0u;", 1, ()),
    ("bf16_half_down", "dropped > 0x8000u ||", "dropped >= 0x8001u && 0 ||", 1, ()),
    ("bf16_nan_unhandled", "if (isnan(f))\n        return", "if (0)\n        return", 1, ()),
    ("rs_wrong_offset", "(uint64_t)rank * recvcount", "(uint64_t)rank", 1, ()),
    ("wrong_index", "up_float(srcs[p], off + i, dtype)", "up_float(srcs[p], i, dtype)", 1, ()),
    ("max_ignores_zero_sign", "return signbit(a) ? b : a;", "return a;", 1, ()),
    ("min_ignores_zero_sign", "return signbit(a) ? a : b;", "return b;", 1, ()),
    ("max_drops_nan", "if (isnan(a) || isnan(b)) return canonical_nan();\n    if (a > b)",
     "if (isnan(a)) return b;\n    if (a > b)", 1, ()),
    ("max_is_min", "if (a > b) return a;", "if (a < b) return a;", 1, ()),
    ("prod_is_sum", "case XO_PROD: return a * b;", "case XO_PROD: return a + b;", 1, ()),
    ("int_max_unsigned", "if (sgn) return ((int32_t)a > (int32_t)b) ? a : b;",
     "if (sgn) return (a > b) ? a : b;", 1, ()),
    ("int_min_signed_for_u32", "return a < b ? a : b;",
     "return ((int32_t)a < (int32_t)b) ? a : b;", 1, ()),
    ("step_init_reads_acc", "float a = init ? x : op_float(op, up_float(acc, i, XO_F32), x);",
     "float a = op_float(op, up_float(acc, i, XO_F32), x);", 1, ()),
    ("step_final_writes_acc", "if (fin) down_float(dst, i, dtype, a);\n            else down_float(acc, i, XO_F32, a);",
     "down_float(acc, i, XO_F32, a);\n            if (fin) down_float(dst, i, dtype, a);", 1, ()),
    ("bf16_accumulates_in_bf16",
     "acc = op_float(fop, acc, up_float(srcs[p], off + i, dtype));",
     "{ acc = op_float(fop, acc, up_float(srcs[p], off + i, dtype)); "
     "if (dtype == XO_BF16) acc = bf16_to_f32(f32_to_bf16(acc)); }", 1, ()),
    ("reverse_fold_order",
     "for (int p = 1; p < nsrc; ++p)\n            acc = op_float(fop, acc, up_float(srcs[p], off + i, dtype));",
     "for (int p = nsrc - 2; p >= 0; --p)\n            acc = op_float(fop, acc, up_float(srcs[p], off + i, dtype));",
     1, ()),
    # binary64 and 8-bit integers
    ("i8_zero_extends", "return dtype == XO_I8 ? (uint32_t)(int32_t)(int8_t)b : (uint32_t)b;",
     "return (uint32_t)b;", 1, ()),
    ("int8_keeps_wrong_byte", "((uint8_t *)base)[i] = (uint8_t)v; }",
     "((uint8_t *)base)[i] = (uint8_t)(v >> 8); }", 1, ()),
    ("i8_max_unsigned", "const int sgn = dtype == XO_I32 || dtype == XO_I8;",
     "const int sgn = dtype == XO_I32;", 1, ()),
    ("f64_accumulates_in_f32", "acc = op_f64(fop, acc, up_f64(srcs[p], off + i));",
     "acc = (double)(float)op_f64(fop, acc, up_f64(srcs[p], off + i));", 1, ()),
    ("f64_avg_in_f32", "if (op == XO_AVG) acc = acc / (double)nsrc;",
     "if (op == XO_AVG) acc = (double)((float)acc / (float)nsrc);", 1, ()),
    ("f64_max_drops_nan",
     "if (isnan(a) || isnan(b)) return canonical_nan64();\n    if (a > b)",
     "if (isnan(a)) return b;\n    if (a > b)", 1, ()),
    ("f64_min_ignores_zero_sign", "if (b < a) return b;\n    return signbit(a) ? a : b;\n}\n\nstatic double op_f64",
     "if (b < a) return b;\n    return b;\n}\n\nstatic double op_f64", 1, ()),
    ("f64_step_rounds_acc", "double a = settle64(op, init ? x : op_f64(op, up_f64(acc, i), x));",
     "double a = settle64(op, init ? x : (double)(float)op_f64(op, up_f64(acc, i), x));", 1, ()),
    # simulated schedules
    ("ring_sendcopy_own_chunk", "const int c = mod_rank(r - 1, G);\n            memcpy(wire[r]",
     "const int c = mod_rank(r, G);\n            memcpy(wire[r]", 1, ()),
    ("ring_reduce_drops_own",
     "hop_reduce(in, elem_at(own[r], LO(c), dtype), elem_at(recv[r], LO(c), dtype),",
     "hop_reduce(in, in, elem_at(recv[r], LO(c), dtype),", 1, ()),
    ("ring_allgather_wrong_slot", "const int c = mod_rank(r - t, G);",
     "const int c = mod_rank(r - t + 1, G);", 1, ()),
    ("ring_recvcopy_does_not_forward", "if (t < G - 1) memcpy(next[r], in, LEN(c) * es);",
     "if (t < G - 1) memcpy(next[r], elem_at(recv[r], LO(r), dtype), LEN(c) * es);", 1, ()),
    ("rhd_keeps_given_half", "const int keep = (r & d) ? lo[r] + half : lo[r];",
     "const int keep = (r & d) ? lo[r] : lo[r] + half;", 1, ()),
    ("rhd_reduces_own_message", "hop_reduce(msg[r ^ d], mine, mine,", "hop_reduce(msg[r], mine, mine,",
     1, ()),
    ("sim_chunks_unaligned", "return (m + XO_SIM_ALIGN - 1) / XO_SIM_ALIGN * XO_SIM_ALIGN;",
     "return m;", 1, ()),
    # further types and AVG
    ("narrow_ties_away", "if (rem > half || (rem == half && (n & 1u))) n += 1;",
     "if (rem >= half) n += 1;", 1, ()),
    ("narrow_flushes_subnormals", "if (n < (1ull << f->mbits)) return sbit | (uint32_t)n;",
     "if (n < (1ull << f->mbits)) return sbit;", 1, ()),
    ("e4m3_overflow_to_nan",
     "const uint32_t overflow = f->has_inf ? (etop << f->mbits) : f->max_finite;",
     "const uint32_t overflow = f->has_inf ? (etop << f->mbits) : f->qnan;", 1, ()),
    ("e5m2_without_infinity", "FMT_E5M2 = {2, 5, 15, 1, 0x7Bu, 0x7Eu};",
     "FMT_E5M2 = {2, 5, 15, 0, 0x7Bu, 0x7Eu};", 1, ()),
    ("f16_wrong_bias", "FMT_F16 = {10, 5, 15, 1, 0x7BFFu, 0x7E00u};",
     "FMT_F16 = {10, 5, 14, 1, 0x7BFFu, 0x7E00u};", 1, ()),
    ("avg_divides_by_p_minus_1", "if (op == XO_AVG) acc = acc / (float)nsrc;",
     "if (op == XO_AVG) acc = acc / (float)(nsrc > 1 ? nsrc - 1 : 1);", 1, ()),
    ("avg_premultiplies",
     "float acc = up_float(srcs[0], off + i, dtype);\n        for (int p = 1; p < nsrc; ++p)\n"
     "            acc = op_float(fop, acc, up_float(srcs[p], off + i, dtype));\n"
     "        if (op == XO_AVG) acc = acc / (float)nsrc;",
     "const float sc = op == XO_AVG ? 1.0f / (float)nsrc : 1.0f;\n"
     "        float acc = op == XO_AVG ? up_float(srcs[0], off + i, dtype) * sc : up_float(srcs[0], off + i, dtype);\n"
     "        for (int p = 1; p < nsrc; ++p)\n"
     "            acc = op_float(fop, acc, op == XO_AVG ? up_float(srcs[p], off + i, dtype) * sc : up_float(srcs[p], off + i, dtype));",
     1, ()),
    ("int64_truncated", "uint64_t acc = up_int64(srcs[0], off + i);",
     "uint64_t acc = (uint32_t)up_int64(srcs[0], off + i);", 1, ()),
    ("i64_max_unsigned", "if (dtype == XO_I64) return ((int64_t)a > (int64_t)b) ? a : b;",
     "if (dtype == XO_I64) return a > b ? a : b;", 1, ()),
    # a fast-math build flushes subnormals (and loads code that sets FTZ/DAZ for
    # the whole process, which is why every mutant runs in a child process)
    ("fast_math_build", None, None, 0, ("-ffast-math",)),
]


def _build_mutant(tmp_path, name, old, new, count, flags):
    text = SRC
    if old is not None:
        assert old in text, f"mutant {name}: anchor text not found in the oracle"
        text = text.replace(old, new) if count == 0 else text.replace(old, new, count)
        # reverse_fold_order starts from the last source instead of the first
        if name == "reverse_fold_order":
            text = text.replace(
                "float acc = up_float(srcs[0], off + i, dtype);\n        for (int p = nsrc - 2;",
                "float acc = up_float(srcs[nsrc - 1], off + i, dtype);\n        for (int p = nsrc - 2;")
    src = tmp_path / f"{name}.c"
    src.write_text(text)
    out = tmp_path / f"lib_{name}.so"
    oracle.build(src, out, extra_flags=list(flags))
    return oracle.Oracle(out)


def _run_pins(name: str, tmp: str) -> int:
    """Child-process body: build the mutant, run the pins, exit 0 if one fails."""
    mutant = next(m for m in MUTANTS if m[0] == name)
    m = _build_mutant(Path(tmp), *mutant)
    for pin in pins.FAST_PINS:
        try:
            pin(m)
        except AssertionError as e:
            print(f"caught by {pin.__name__}: {str(e)[:120]}")
            return 0
    print("survived")
    return 1


@pytest.mark.parametrize("mutant", MUTANTS, ids=lambda m: m[0])
def test_pins_catch_mutant(tmp_path, mutant):
    name = mutant[0]
    r = subprocess.run([sys.executable, __file__, name, str(tmp_path)], capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 0, f"mutant {name}: {r.stdout.strip()} {r.stderr[-500:]}"


if __name__ == "__main__":
    sys.path.insert(0, str(ROOT / "tests"))
    sys.exit(_run_pins(sys.argv[1], sys.argv[2]))
