"""The fp64 oracle against its pins (CPU only), and the pins against planted
mistakes: each mutant is a copy of the oracle's C source with one plausible
error (a wrong index, a dropped term, a swapped operand), compiled to a
temporary library; at least one pin must reject every mutant."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle_pins as pins

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(oracle_lib, pin):
    pin(oracle_lib)


MUTANTS = {
    "head_map_modulo": ("const int g = h / G;", "const int g = h % n_kv_heads;"),
    "slot_index": ("(size_t)(t % page_size) * row + (size_t)g * head_dim;\n        double dot",
                   "(size_t)((t + 1) % page_size) * row + (size_t)g * head_dim;\n        double dot"),
    "page_table_row_stride": ("page_table[(size_t)b * max_pages_per_seq + t / page_size];\n        const uint16_t *kt",
                              "page_table[(size_t)b * (t / page_size + 1) + t / page_size];\n        const uint16_t *kt"),
    "no_max_subtraction": ("scores[t] = exp(scores[t] - m);", "scores[t] = exp(scores[t]);"),
    "scale_dropped": ("scores[t] = scale * dot;", "scores[t] = dot;"),
    "no_normaliser": ("out[d] /= z;", "out[d] /= 1.0;"),
    "v_from_k_pool": ("const uint16_t *vt = v_pages", "const uint16_t *vt = k_pages"),
    "q_head_of_kv": ("const uint16_t *qh = q + ((size_t)b * n_q_heads + h) * head_dim;",
                     "const uint16_t *qh = q + ((size_t)b * n_q_heads + g * G) * head_dim;"),
    "last_token_dropped": ("for (int t = 0; t < L; ++t) {\n        const int32_t p = page_table[(size_t)b * max_pages_per_seq + t / page_size];\n        const uint16_t *vt",
                           "for (int t = 0; t < L - 1; ++t) {\n        const int32_t p = page_table[(size_t)b * max_pages_per_seq + t / page_size];\n        const uint16_t *vt"),
    "bf16_widen_shift": ("uint32_t bits = (uint32_t)h << 16;", "uint32_t bits = (uint32_t)h << 15;"),
    "gather_v_from_k": ("memcpy(v_out + dst, v_pages + src", "memcpy(v_out + dst, k_pages + src"),
    "append_slot": ("(size_t)(pos % page_size) * row;\n        memcpy(k_pages",
                    "(size_t)((pos + 1) % page_size) * row;\n        memcpy(k_pages"),
    "gemm_transposed_w": ("vdo_bf16_to_f64(w[(size_t)n * K + k]);", "vdo_bf16_to_f64(w[(size_t)k * N + n]);"),
    "gemm_k_off_by_one": ("for (int k = 0; k < K; ++k)\n            acc +=", "for (int k = 1; k < K; ++k)\n            acc +="),
    "append_no_skip": ("if (pos < 0 || pos >= max_pages_per_seq * page_size)\n            continue;",
                       "if (pos < 0)\n            continue;"),
}


def _build_mutant(tmp_path, name, old, new):
    src = open(os.path.join(os.path.dirname(pins.__file__), "..", "oracle", "vdo_oracle.c")).read()
    assert src.count(old) == 1, "mutation site for %s not unique/found" % name
    path = tmp_path / ("%s.c" % name)
    path.write_text(src.replace(old, new))
    lib = tmp_path / ("lib%s.so" % name)
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-o", str(lib),
                    str(path), "-lm"], check=True, capture_output=True)
    return str(lib)


class _MutantOracle:
    """Same Python surface as the oracle package, bound to a mutant library."""

    def __init__(self, libpath):
        import oracle
        self._o = oracle
        self._lib = ctypes.CDLL(libpath)
        proto = oracle._load()
        for fn in ("vdo_decode_attn_f64", "vdo_decode_attn_rows_f64", "vdo_gather",
                   "vdo_kv_append", "vdo_gemm_f64", "vdo_softmax_f64", "vdo_max_threads"):
            getattr(self._lib, fn).argtypes = getattr(proto, fn).argtypes
            getattr(self._lib, fn).restype = getattr(proto, fn).restype

    def __getattr__(self, name):
        fn = getattr(self._o, name)

        def call(*a, **k):
            saved = self._o._lib
            self._o._lib = self._lib
            try:
                return fn(*a, **k)
            finally:
                self._o._lib = saved
        return call


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(tmp_path, oracle_lib, name):
    old, new = MUTANTS[name]
    mut = _MutantOracle(_build_mutant(tmp_path, name, old, new))
    failed = []
    for pin in pins.ALL_PINS:
        try:
            with np.errstate(all="ignore"):
                pin(mut)
        except (AssertionError, RuntimeError, IndexError, ValueError):
            failed.append(pin.__name__)
    assert failed, "no pin rejects mutant %s" % name


def test_rows_function_equals_full_oracle(oracle_lib):
    """The oracle's sampled-row function (used where the full output is too
    slow on the CPU) returns exactly the full oracle's rows: same arithmetic,
    same order, bit for bit."""
    import numpy as np
    from workloads import Workload, bits, make_case
    w = Workload("custom", 5, 32, 8, 128, 16, "fixed", (1, 17, 300, 0, 1000))
    c = make_case(w, seed=8, fill="nan")
    args = (bits(c["q"]), bits(c["k_pages"]), bits(c["v_pages"]), c["page_table"].numpy(),
            c["seq_lens"].numpy())
    full = oracle_lib.decode_attn(*args, c["scale"])
    sel_b = np.array([0, 1, 2, 2, 3, 4, 4], dtype=np.int32)
    sel_h = np.array([0, 31, 5, 6, 9, 0, 31], dtype=np.int32)
    rows = oracle_lib.decode_attn_rows(*args, c["scale"], sel_b, sel_h)
    assert np.array_equal(rows, full[sel_b, sel_h])
