"""Mutation check of the oracle's pins: each plausible mistake below is
planted in a copy of the oracle source, and the pin module that guards that
part of the method must then fail.  A mistake no pin catches would mean the
oracle is not tied down where the paper or the mathematics fixes it.

Each case copies oracle/, synthetic/ and tests/ into a temporary directory,
edits the copy of cpes_oracle.c, and runs the named pin test there with
pytest (-x: the first failure is enough)."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# (name, text in cpes_oracle.c, replacement, pin test that must fail)
MUTANTS = [
    ("philox multiplier", "#define PHILOX_M0 0xD2511F53u", "#define PHILOX_M0 0xD2511F55u",
     "test_oracle_philox.py::test_philox_matches_torch_and_rocrand"),
    ("cosine and sine swapped", "return (float)(rho * ((t & 1) ? s : c));",
     "return (float)(rho * ((t & 1) ? c : s));",
     "test_oracle_normal.py::test_normal_equals_rounded_product"),
    ("uniform grid shifted to [0, 1)", "return (double)((x >> 8) + 1u) * 0x1p-24;",
     "return (double)((x >> 8) + 0u) * 0x1p-24 + 0x1p-25;",
     "test_oracle_normal.py::test_uniform_identities"),
    ("second-quadrant cosine sign", "case 1: *cos_out = -sr; *sin_out = cr;  break;",
     "case 1: *cos_out = sr; *sin_out = cr;  break;",
     "test_oracle_normal.py::test_angle_diagonals"),
    ("angle word of the second pair", "uint32_t b = (t < 2) ? x[1] : x[3];", "uint32_t b = (t < 2) ? x[1] : x[2];",
     "test_oracle_normal.py::test_normal_equals_rounded_product"),
    ("perturbation ignores the sign", "float scale = (float)sign * sigma; /* exact: a sign flip */",
     "float scale = sigma;",
     "test_oracle_ops.py::test_perturb_is_one_fp32_fma"),
    ("paper scale divided by sigma", ": (double)alpha / (double)n;", ": (double)alpha / ((double)n * (double)sigma);",
     "test_oracle_ops.py::test_update_brute_force_fp32"),
    ("mirrored sign dropped from the coefficient", "coef[u] += (double)signs[i] * (double)rnorm[i];",
     "coef[u] += (double)rnorm[i];",
     "test_oracle_ops.py::test_update_brute_force_fp32"),
    ("update noise index ignores the window start", "acc += coef[u] * (double)orc_normal(useed[u], j0 + j);",
     "acc += coef[u] * (double)orc_normal(useed[u], j);",
     "test_oracle_ops.py::test_update_brute_force_fp32"),
    ("sample instead of population std", "double s = sqrt(ss / (double)count);",
     "double s = sqrt(ss / (double)(count - 1));",
     "test_oracle_ops.py::test_z_normalisation_matches_numpy"),
    ("ties not averaged in ranks", "double a = (double)less + 0.5 * (double)(equal - 1);",
     "double a = (double)less + 0.5 * (double)equal;",
     "test_oracle_ops.py::test_rank_normalisation_matches_scipy"),
    ("bucket of the element instead of its image",
     "return (int32_t)((e * (unsigned __int128)(uint32_t)K) / (unsigned __int128)(uint64_t)d);",
     "return (int32_t)(((unsigned __int128)(uint64_t)i * (unsigned __int128)(uint32_t)K) / "
     "(unsigned __int128)(uint64_t)d + 0*e);",
     "test_oracle_partition.py::test_permutation_is_replayable_and_seeded"),
    ("master restore not exact", "store_w(w, dtype, i, ((const float*)aux)[j]);",
     "store_w(w, dtype, i, ((const float*)aux)[j] * 1.0000001f);",
     "test_oracle_ops.py::test_bf16_rounding_matches_torch"),
    ("replay restore adds instead of subtracting", "float scale = -(float)sign * sigma;",
     "float scale = (float)sign * sigma;",
     "test_oracle_ops.py::test_replay_restore_is_not_an_identity_but_is_bounded"),
]


def _copy_tree(dst):
    ignore = shutil.ignore_patterns("*.so", "__pycache__", "*.pyc")
    for d in ("oracle", "synthetic", "tests"):
        shutil.copytree(os.path.join(ROOT, d), os.path.join(dst, d), ignore=ignore)


@pytest.mark.parametrize("name,old,new,pin", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_fails_its_pin(tmp_path, name, old, new, pin):
    _copy_tree(str(tmp_path))
    src = tmp_path / "oracle" / "cpes_oracle.c"
    text = src.read_text()
    assert text.count(old) == 1, f"mutation site of '{name}' not found once in the oracle"
    src.write_text(text.replace(old, new))
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                          os.path.join("tests", pin)], cwd=str(tmp_path), capture_output=True, text=True,
                         timeout=600)
    tail = res.stdout[-1500:]
    assert res.returncode == 1 and " failed" in tail, f"'{name}' survived {pin}:\n{tail}\n{res.stderr[-800:]}"
