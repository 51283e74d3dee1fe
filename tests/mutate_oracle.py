"""Plants one mistake at a time in a copy of the oracle and checks that its
pins catch it. Run by hand (`python tests/mutate_oracle.py`); pytest does
not collect it. Each mutant is a plausible slip in the oracle's arithmetic
(a flipped comparison, a swapped operand or index, a dropped step); the
oracle's CPU tests (Philox vectors, brute-force sampler checks, closed forms
of the buffer policy, the independent replay and the property runs) must
fail on every one, except mutants that cannot change any output, which are
listed with the reason. Works in a temporary directory; the repository is
not touched."""
import os
import shutil
import subprocess
import sys
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PINS = ["tests/test_oracle_philox.py", "tests/test_oracle_sampler.py", "tests/test_oracle_buffer.py",
        "tests/test_oracle_subnormal.py", "tests/test_oracle_fuzz.py"]

# (label, text in oracle.c, replacement)
MUTANTS = [
    ("decay applied to sampled slots", "if (!sampled) c->S_E[s]", "if (sampled) c->S_E[s]"),
    ("S_A += 1 on hits", "      if (c->mask[i] == 2) {", "      if (c->mask[i] == 1) {"),
    ("eviction at S_E <= alpha", "if (c->S_E[s] < c->alpha)", "if (c->S_E[s] <= c->alpha)"),
    ("candidates by S_A ascending", "if (sx != sy) return sx > sy ? -1 : 1;", "if (sx != sy) return sx < sy ? -1 : 1;"),
    ("slot gets the evicted node's S_E", "c->S_E[s] = oldSA[i];", "c->S_E[s] = oldSE[i];"),
    ("evicted node's S_A reset to 0", "c->S_A[e] = oldSE[i];", "c->S_A[e] = 0.0f;"),
    ("replacement keeps its S_A", "c->S_A[r] = -1.0f;               /* replacement", "(void)0;  /* replacement"),
    ("Philox: wrong key word in a round", "uint32_t y0 = hi1 ^ x1 ^ k0;", "uint32_t y0 = hi1 ^ x1 ^ k1;"),
    ("Philox: wrong Weyl constant", "k1 += W1;", "k1 += W0;"),
    ("sampler keeps the largest keys", "sel[i] = (int64_t)(keybuf[i] & 0xffffffffu);",
     "sel[i] = (int64_t)(keybuf[d - 1 - i] & 0xffffffffu);"),
    ("chosen positions not re-sorted", "while (p > 0 && sel[p - 1] > x)", "while (0)"),
    ("counter words v and t swapped", "(uint32_t)(j / 4), (uint32_t)v, (uint32_t)c->t, (uint32_t)k}",
     "(uint32_t)(j / 4), (uint32_t)c->t, (uint32_t)v, (uint32_t)k}"),
    ("key word index off by one", "((uint64_t)words[j % 4] << 32)", "((uint64_t)words[(j + 1) % 4] << 32)"),
    ("rank by degree ascending", "if (dx != dy) return dx > dy ? -1 : 1;", "if (dx != dy) return dx < dy ? -1 : 1;"),
    ("rank ties by global id descending", "return gx < gy ? -1 : gx > gy;", "return gx > gy ? -1 : gx < gy;"),
    ("alpha with one product too many", "i < a->delta; i++) al = al * a->gamma;",
     "i <= a->delta; i++) al = al * a->gamma;"),
    ("new nodes not checked against F", "      if (c->pos[u] >= 0) continue;", "      (void)0;"),
    ("short-candidate eviction by S_E descending", "if (ex != ey) return ex < ey ? -1 : 1;",
     "if (ex != ey) return ex > ey ? -1 : 1;"),
    ("decay flushes subnormal products to zero", "if (!sampled) c->S_E[s] = c->S_E[s] * c->a.gamma;",
     "if (!sampled) { float x_ = c->S_E[s] * c->a.gamma; c->S_E[s] = x_ < 1.17549435e-38f ? 0.0f : x_; }"),
]
# (label, extra gcc flags): the unchanged source built another way. With gcc,
# -ffast-math also links crtfastmath.o, which sets flush-to-zero and
# denormals-are-zero for the thread that loads the library.
FLAG_MUTANTS = [
    ("built with -ffast-math (flush to zero)", ["-ffast-math"]),
]
# mutants that cannot change any output
EQUIVALENT = [
    # after one step every slot has S_E >= gamma >= gamma^Delta = alpha, so a
    # round after step 0 would find no slot below alpha
    ("round also after step 0", "if (!(t > 0 && t % c->a.delta == 0))", "if (!(t % c->a.delta == 0))"),
]


def run(label, old, new, tmp, flags=()):
    tree = os.path.join(tmp, "tree")
    shutil.rmtree(tree, ignore_errors=True)
    os.makedirs(tree)
    for d in ("tests", "oracle", "synth"):
        shutil.copytree(os.path.join(ROOT, d), os.path.join(tree, d),
                        ignore=shutil.ignore_patterns("*.so", "__pycache__", ".hypothesis"))
    src = os.path.join(tree, "oracle", "oracle.c")
    text = open(src).read()
    if old is not None:
        if text.count(old) != 1:
            raise SystemExit("mutant %r: the text to replace occurs %d times" % (label, text.count(old)))
        open(src, "w").write(text.replace(old, new))
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off"] + list(flags) +
                          [src, "-o", os.path.join(tree, "oracle", "liboracle.so")])
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-p", "no:warnings"]
                       + PINS, cwd=tree, capture_output=True, text=True, timeout=900)
    return r.returncode != 0, (r.stdout.strip().splitlines() or [""])[-1]


def main():
    survivors = []
    with tempfile.TemporaryDirectory() as tmp:
        for label, old, new in MUTANTS:
            caught, last = run(label, old, new, tmp)
            print("%-45s %s  (%s)" % (label, "caught" if caught else "SURVIVED", last), flush=True)
            if not caught:
                survivors.append(label)
        for label, flags in FLAG_MUTANTS:
            caught, last = run(label, None, None, tmp, flags)
            print("%-45s %s  (%s)" % (label, "caught" if caught else "SURVIVED", last), flush=True)
            if not caught:
                survivors.append(label)
        for label, old, new in EQUIVALENT:
            caught, last = run(label, old, new, tmp)
            print("%-45s %s  (%s; cannot change any output)" % (label, "caught" if caught else "not caught", last),
                  flush=True)
    if survivors:
        raise SystemExit("mutants not caught: %s" % ", ".join(survivors))


if __name__ == "__main__":
    main()
