"""The oracle's pins are sensitive: each plausible mistake planted in a copy of
the oracle source (a dropped term, a wrong index, a flipped comparison) must
make the pin suite fail.  Mutants are built and run on the CPU only."""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PIN_FILES = ["tests/test_oracle_fuse.py", "tests/test_oracle_decode.py",
             "tests/test_oracle_evict.py", "tests/test_oracle_offsets.py", "tests/test_oracle_run.py"]

MUTANTS = {
    "drop_decay": ("score_out[(size_t)l * T + j] = gamma * prev + psum[j];",
                   "score_out[(size_t)l * T + j] = prev + psum[j];"),
    "scale_by_d": ("sm_scale = 1.0 / sqrt((double)d);", "sm_scale = 1.0 / (double)d;"),
    "gqa_modulo": ("(int32_t)(((int64_t)h * Hkv) / Hq)", "(int32_t)(h % Hkv)"),
    "no_normalise": ("                s[j] /= z;\n", "\n"),
    "new_key_from_cache": (": ld(k_new, dtype, nb + c);", ": ld(k_cache, dtype, cb + (size_t)j * d + c);"),
    "new_slot_nonzero": ("double prev = (j < len) ? score_in[(size_t)l * cap + j] : 0.0;",
                         "double prev = (j < len) ? score_in[(size_t)l * cap + j] : 1.0;"),
    "mean_divisor": ("double mean = sum / (double)count;", "double mean = sum / (double)(count + 1);"),
    "anchor_subtracted": ("mean += ld(anchor,", "mean -= ld(anchor,"),
    "topn_ascending": ("if (x->score > y->score)", "if (x->score < y->score)"),
    "recent_off_by_one": ("c.pos >= next_pos - M", "c.pos > next_pos - M"),
    "sink_off_by_one": ("c.pos < n_sink", "c.pos <= n_sink"),
    "eq3_round_up": ("((int64_t)L_a * te) / t_total_ms", "((int64_t)L_a * te + t_total_ms - 1) / t_total_ms"),
    "groups_not_min": ("int64_t g = seg[i].lt < len ? seg[i].lt : len;", "int64_t g = len;"),
}


# Mistakes planted in the Python driver (oracle/__init__.py): each a list of
# (old, new) replacements.
PY_MUTANTS = {
    # the selection ranks the scores from before this step's Eq. (6) update
    "evict_before_fold": [
        ("        out, s, p, _ = decode_step(q, k_new, v_new, self.k, self.v, self.score, self.pos,",
         "        pre = self.score.copy()\n"
         "        out, s, p, _ = decode_step(q, k_new, v_new, self.k, self.v, self.score, self.pos,"),
        ("            self.evict()\n        return out", "            self.evict(pre)\n        return out"),
        ("    def evict(self):\n        keep, nl = evict_select(self.score, self.pos,",
         "    def evict(self, pre=None):\n        keep, nl = evict_select(self.score if pre is None else pre, self.pos,"),
    ],
    # the trigger tested on the step index before it is advanced (t % interval)
    "interval_t_mod": [
        ("        self.t += 1\n        if self.t % self.interval == 0 and self.len > self.budget:\n"
         "            self.evict()\n",
         "        if self.t % self.interval == 0 and self.len > self.budget:\n"
         "            self.evict()\n        self.t += 1\n"),
    ],
    # scores compacted, positions left where they were
    "gather_score_not_pos": [("        self.pos[:, :nl] = gather_rows(self.pos, keep)\n", "")],
    # bfloat16 storage by truncation instead of nearest-even
    "round_truncate": [("((b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16))",
                        "(b >> np.uint32(16))")],
    # Eq. 7-8 gather applied along the head axis of K/V
    "gather_head_axis": [("np.stack([x[l][:, keep[l], :] for l in range(L)])",
                          "np.stack([x[l][keep[l] % x.shape[1]] for l in range(L)])")],
}


@pytest.mark.parametrize("name", sorted(PY_MUTANTS))
def test_pins_catch_planted_driver_mistake(name, tmp_path):
    src = open(os.path.join(ROOT, "oracle", "__init__.py")).read()
    for old, new in PY_MUTANTS[name]:
        assert src.count(old) == 1, f"mutation site for {name} is not unique: {old!r}"
        src = src.replace(old, new)
    pkg = tmp_path / "oracle"
    pkg.mkdir()
    (pkg / "__init__.py").write_text(src)
    (pkg / "voxzip_oracle.c").write_text(open(os.path.join(ROOT, "oracle", "voxzip_oracle.c")).read())
    lib = str(tmp_path / "liboracle.so")
    oracle.build(out=lib)
    env = dict(os.environ, VOXZIP_ORACLE_LIB=lib, OMP_NUM_THREADS="2")
    # the mutant package is imported before pytest, so every test module gets it
    boot = (f"import sys; sys.path.insert(0, {str(tmp_path)!r}); import oracle; "
            f"assert oracle.__file__.startswith({str(tmp_path)!r}); import pytest; "
            f"sys.exit(pytest.main(['-x', '-q', '-p', 'no:cacheprovider', *{PIN_FILES!r}]))")
    r = subprocess.run([sys.executable, "-c", boot], cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    # a pin must fail (not the import of the mutant, which also exits with 1)
    assert r.returncode == 1 and " failed" in r.stdout, \
        f"mutant {name} survived the pins:\n{r.stdout[-2000:]}{r.stderr[-2000:]}"


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(os.path.join(ROOT, "oracle", "voxzip_oracle.c")).read()
    assert src.count(old) == 1, f"mutation site for {name} is not unique"
    mutant_src = tmp_path / "mutant.c"
    mutant_src.write_text(src.replace(old, new))
    lib = str(tmp_path / "libmutant.so")
    oracle.build(out=lib, src=str(mutant_src))
    env = dict(os.environ, VOXZIP_ORACLE_LIB=lib, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", *PIN_FILES],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 1, f"mutant {name} survived the pins:\n{r.stdout[-2000:]}"
