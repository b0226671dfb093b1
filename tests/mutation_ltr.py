"""Mutation check of the SJF (LTR+) oracle (a CPU tool, not collected by pytest).

Each entry plants one plausible mistake in a copy of oracle/tas_oracle.c and
runs the LTR+, replay and hand-worked pins against that copy; every mutation
must make at least one of them fail. The repository's own oracle is left
untouched. Usage: python tests/mutation_ltr.py
"""
import os
import shutil
import subprocess
import sys
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# name: (text in the oracle, its mutated form)
MUTATIONS = {
    "no_reset_when_served": (
        "                    if (!q->promoted) {\n                        q->starve = 0;\n",
        "                    if (!q->promoted) {\n                        ;\n"),
    "threshold_off_by_one": ("++q->starve >= I->ltr_s", "++q->starve > I->ltr_s"),
    "promotion_order_ignored": ("q->promo_key = (iters + 1) - PROMOTED_OFFSET;",
                                "q->promo_key = -PROMOTED_OFFSET;"),
    "lifo_promotion": ("q->promo_key = (iters + 1) - PROMOTED_OFFSET;",
                       "q->promo_key = -(iters + 1) - PROMOTED_OFFSET;"),
    "quantum_never_spent": ("} else if (--q->starve == 0) {", "} else if (0) {"),
    "quantum_one_short": ("} else if (--q->starve == 0) {", "} else if (--q->starve <= 1) {"),
    "demotion_keeps_count": (
        "                        q->promoted = 0; /* the quantum is spent */",
        "                        q->promoted = 0; q->starve = I->ltr_s - 1;"),
    "promoted_key_is_sjf": ("        return q->promoted ? q->promo_key : I->D[r];",
                            "        return I->D[r];"),
    "starve_counts_promoted": ("} else if (!q->promoted && ++q->starve >= I->ltr_s) {",
                               "} else if (++q->starve >= I->ltr_s) {"),
}
TESTS = ["tests/test_oracle_pins.py", "tests/test_oracle_invariants.py",
         "tests/test_oracle_comparators.py"]


def main() -> int:
    src = open(os.path.join(ROOT, "oracle", "tas_oracle.c")).read()
    missed = []
    for name, (a, b) in MUTATIONS.items():
        assert src.count(a) == 1, f"{name}: the oracle text it mutates changed"
        with tempfile.TemporaryDirectory(prefix=f"mut_{name}_") as d:
            shutil.copytree(os.path.join(ROOT, "oracle"), os.path.join(d, "oracle"),
                            ignore=shutil.ignore_patterns("*.so", "__pycache__"))
            with open(os.path.join(d, "oracle", "tas_oracle.c"), "w") as f:
                f.write(src.replace(a, b))
            os.symlink(os.path.join(ROOT, "paper_2606_18431_amd"),
                       os.path.join(d, "paper_2606_18431_amd"))
            shutil.copytree(os.path.join(ROOT, "tests"), os.path.join(d, "tests"),
                            ignore=shutil.ignore_patterns("__pycache__"))
            shutil.copy(os.path.join(ROOT, "pytest.ini"), d)
            r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                                "-m", "not gpu", "-k", "ltr or replay or hand_worked"] + TESTS,
                               cwd=d, capture_output=True, text=True, timeout=1800)
        caught = r.returncode != 0
        first = next((ln for ln in r.stdout.splitlines() if "FAILED" in ln), "")
        print(f"{name}: {'caught' if caught else 'MISSED'} {first}", flush=True)
        if not caught:
            missed.append(name)
    print(f"{len(MUTATIONS) - len(missed)} of {len(MUTATIONS)} mutations caught")
    return 1 if missed else 0


if __name__ == "__main__":
    sys.exit(main())
