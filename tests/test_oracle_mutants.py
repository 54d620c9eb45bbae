"""The oracle pins must catch plausible mistakes.

Each case plants one mistake in a private copy of the oracle's C source (a
dropped term, a wrong sign or index, a wrong seed, a wrong readout order, ...),
compiles it, and runs the pin suite against it in a subprocess.  The suite must
fail for every mutant.  Nothing here touches the product library or a GPU.
"""
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "bdgdn_oracle.c")

NOISY_LOOPS = """        for (long l = p0; l < p1; ++l)
            gdr_step(Sn, d->dk, d->dv, row_qk(kn, d, l, h), row_v(vn, d, l, h),
                     gate_at(gn, d, l, h), gate_at(betan, d, l, h), u);
        for (long l = p0; l < p1; ++l)       /* block-end readout */
            readout(Sn, d->dk, d->dv, row_qk(qn, d, l, h), d->scale, row_o(on, d, l, h));"""
NOISY_PER_POSITION = """        for (long l = p0; l < p1; ++l) {
            gdr_step(Sn, d->dk, d->dv, row_qk(kn, d, l, h), row_v(vn, d, l, h),
                     gate_at(gn, d, l, h), gate_at(betan, d, l, h), u);
            readout(Sn, d->dk, d->dv, row_qk(qn, d, l, h), d->scale, row_o(on, d, l, h));
        }"""
CLEAN_STEP = """            gdr_step(S, d->dk, d->dv, row_qk(k, d, t, h), row_v(v, d, t, h),
                     gate_at(g, d, t, h), gate_at(beta, d, t, h), u);
            readout(S, d->dk, d->dv, row_qk(q, d, t, h), d->scale, row_o(o, d, t, h));"""
CLEAN_READ_FIRST = """            readout(S, d->dk, d->dv, row_qk(q, d, t, h), d->scale, row_o(o, d, t, h));
            gdr_step(S, d->dk, d->dv, row_qk(k, d, t, h), row_v(v, d, t, h),
                     gate_at(g, d, t, h), gate_at(beta, d, t, h), u);"""

MUTANTS = {
    "no_gating_decay": ("for (int i = 0; i < dk * dv; ++i) S[i] *= alpha;", ";"),
    "alpha_sign": ("const double alpha = exp(g);", "const double alpha = exp(-g);"),
    "prediction_sign": ("u[j] = beta * (v[j] - acc);", "u[j] = beta * (v[j] + acc);"),
    "dropped_beta": ("u[j] = beta * (v[j] - acc);", "u[j] = (v[j] - acc);"),
    "write_factor": ("S[i * dv + j] += k[i] * u[j];", "S[i * dv + j] += 0.5 * k[i] * u[j];"),
    "readout_index": ("acc += S[i * dv + j] * q[i];", "acc += S[i * dv + j] * q[(i + 1) % dk];"),
    "prediction_index": ("acc += S[i * dv + j] * k[i];", "acc += S[i * dv + j] * k[(i + 1) % dk];"),
    "noisy_seed_zero": ("        memcpy(Sn, S, ssz * sizeof(double));",
                        "        memset(Sn, 0, ssz * sizeof(double));"),
    "noisy_not_reset": ("        memcpy(Sn, S, ssz * sizeof(double));",
                        "        if (p0 == r0) memcpy(Sn, S, ssz * sizeof(double));"),
    "noisy_per_position_readout": (NOISY_LOOPS, NOISY_PER_POSITION),
    "clean_read_before_write": (CLEAN_STEP, CLEAN_READ_FIRST),
    "noisy_uses_clean_keys": ("row_qk(kn, d, l, h), row_v(vn, d, l, h)",
                              "row_qk(k, d, l, h), row_v(vn, d, l, h)"),
    "clean_uses_noisy_gates": ("gate_at(g, d, t, h), gate_at(beta, d, t, h)",
                               "gate_at(gn, d, t, h), gate_at(beta, d, t, h)"),
    "gva_mapping": ("int hq = h / (d->h_v / d->h_qk);", "int hq = h % d->h_qk;"),
    "doc_state_not_reset": ("                else memset(S, 0, ssz * sizeof(double));",
                            "                else if (n == 0) memset(S, 0, ssz * sizeof(double));"),
    "denoise_writes_pool": (
        "                readout(Sn, dk, dv, row_qk(q, &d, l, h), scale, row_o(o, &d, l, h));",
        "                readout(Sn, dk, dv, row_qk(q, &d, l, h), scale, row_o(o, &d, l, h));\n"
        "            memcpy((double *)pool + ((size_t)s * h_v + h) * ssz, Sn, ssz * sizeof(double));"),
    "record_after_update": (
        "                if (i >= 0)   /* the state before position p */\n"
        "                    memcpy(states + (((size_t)r * n_rec + i) * h_v + h) * ssz, S, ssz * sizeof(double));\n"
        "                gdr_step(S, dk, dv, row_qk(k, &d, t, h), row_v(v, &d, t, h),\n"
        "                         gate_at(g, &d, t, h), gate_at(beta, &d, t, h), u);\n",
        "                gdr_step(S, dk, dv, row_qk(k, &d, t, h), row_v(v, &d, t, h),\n"
        "                         gate_at(g, &d, t, h), gate_at(beta, &d, t, h), u);\n"
        "                if (i >= 0)\n"
        "                    memcpy(states + (((size_t)r * n_rec + i) * h_v + h) * ssz, S, ssz * sizeof(double));\n"),
    "accept_offset_shift": ("states + (((size_t)r * n_rec + accept[r]) * h_v + h) * ssz",
                            "states + (((size_t)r * n_rec + (accept[r] + 1) % n_rec) * h_v + h) * ssz"),
    "conv_noisy_block_rule": ("sn += w[c * W + i] * (src >= blk ? xn[src * D + c] : x[src * D + c]);",
                              "sn += w[c * W + i] * (src > blk ? xn[src * D + c] : x[src * D + c]);"),
    "conv_reads_across_documents": ("        if (src < a) break;\n        sc += w[c * W + i] * x[src * D + c];",
                                    "        if (src < 0) break;\n        sc += w[c * W + i] * x[src * D + c];"),
    "conv_silu_grad": ("return sg * (1.0 + p * (1.0 - sg));", "return sg;"),
    "conv_dw_misses_noisy": ("                        dw[c * W + i] += gn * xn[src * D + c];",
                             "                        dw[c * W + i] += 0.0 * gn * xn[src * D + c];"),
    "bwd_drops_prediction_term": ("dk[a] -= acc;", "dk[a] -= 0.0 * acc;"),
    "bwd_gate_grad_previous_state": ("dgate += dsp * Spre[a * dvv + j];",
                                     "dgate += dsp * Spre[a * dvv + j] / decay;"),
    "bwd_carry_without_gate": ("dS[a * dvv + j] = decay * dsp;", "dS[a * dvv + j] = dsp;"),
    "bwd_no_noisy_injection": ("for (size_t e = 0; e < ssz; ++e) dS[e] += dSn[e];", ";"),
    "bwd_noisy_reads_first_state": ("const double *Send = Sst + (p1 - p0 - 1) * ssz;",
                                    "const double *Send = Sst;"),
    "bwd_drops_step_size_grad": ("*db += dbeta;", "*db += 0.0 * dbeta;"),
    "bwd_write_without_step_size": ("acc += dS[a * dvv + j] * beta * u[j];", "acc += dS[a * dvv + j] * u[j];"),
    "bwd_seed_of_previous_block": ("const double *seed = ck + b * ssz;",
                                   "const double *seed = ck + (b > 0 ? b - 1 : 0) * ssz;"),
    "commit_skips_last_token": ("for (long t = (long)r * L; t < (long)r * L + L; ++t) {",
                                "for (long t = (long)r * L; t < (long)r * L + L - 1; ++t) {"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not unique"
    with tempfile.TemporaryDirectory() as td:
        path = os.path.join(td, "mutant.c")
        lib = os.path.join(td, "libmutant.so")
        open(path, "w").write(src.replace(old, new))
        subprocess.run(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-o", lib, path, "-lm"],
                       check=True, capture_output=True)
        env = dict(os.environ, BDGDN_ORACLE_LIB=lib, OMP_NUM_THREADS="2")
        r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                            os.path.join(ROOT, "tests", "test_oracle_pins.py")],
                           cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
        assert r.returncode != 0, f"mutant {name} passed every pin:\n{r.stdout[-2000:]}"
