"""Writes the exact-rational fixtures in this directory.

Run:  python tests/golden/make_golden.py

Nothing here calls the HIP path, and nothing calls the oracle either: every
value is derived in exact rational arithmetic (fractions.Fraction) from the
paper's definitions on inputs whose attention has a closed form.

uniform_block_mass.txt
    Q = 0 makes every admissible score equal, so row i of the causal softmax
    (Section 3, eq. recurrent_attention) is uniform: A_ij = 1/(i+1) for
    j <= i.  The block mass of Section 5.1, eq. (block_attention_mass), is then
        r_qb = (1/B) sum_{i in I_q} |{j in I_b : j <= i}| / (i + 1).
    One line per (n, B, qb, kb): the exact value as p/q.

uniform_support.txt
    The arg-min support of Section 5.1, eq. (block_working_set), on those
    uniform masses, found by exhaustive search over all subsets of the
    admissible blocks in exact arithmetic, for the thresholds listed.  When
    several minimum-size subsets reach the threshold, the one whose mass is
    largest and, among those, whose sorted block list is smallest
    lexicographically, is recorded (ties broken by lower block index).  The
    last column is 1 when some prefix of the descending order hits the
    threshold exactly (c_k == tau * total): floating point may then round
    either way, so such rows pin only the exact-arithmetic path.
"""

from __future__ import annotations

import itertools
import os
from fractions import Fraction

HERE = os.path.dirname(os.path.abspath(__file__))
CASES = [(12, 3), (16, 4), (24, 3), (32, 4)]
TAUS = [Fraction(1, 4), Fraction(1, 2), Fraction(3, 4), Fraction(9, 10), Fraction(19, 20), Fraction(1, 1)]


def uniform_mass(n, B):
    nb = n // B
    r = [[Fraction(0)] * nb for _ in range(nb)]
    for qb in range(nb):
        for kb in range(nb):
            tot = Fraction(0)
            for i in range(qb * B, (qb + 1) * B):
                cnt = sum(1 for j in range(kb * B, (kb + 1) * B) if j <= i)
                tot += Fraction(cnt, i + 1)
            r[qb][kb] = tot / B
    return r


def best_support(v, qb, tau):
    cand = list(range(qb + 1))
    total = sum(v[b] for b in cand)
    for k in range(0, qb + 2):
        hits = [c for c in itertools.combinations(cand, k) if sum(v[b] for b in c) >= tau * total]
        if hits:
            best = max(sum(v[b] for b in c) for c in hits)
            tops = sorted(sorted(c) for c in hits if sum(v[b] for b in c) == best)
            return tops[0]
    raise AssertionError


def exact_hit(v, qb, tau):
    desc = sorted(v[: qb + 1], reverse=True)
    total = sum(desc)
    c = Fraction(0)
    for x in [Fraction(0)] + desc:
        c += x
        if c == tau * total:
            return 1
    return 0


def main():
    with open(os.path.join(HERE, "uniform_block_mass.txt"), "w") as f:
        f.write("# n B qb kb r_qb   (Q = 0: uniform causal attention; Section 5.1, "
                "eq. block_attention_mass; exact)\n")
        for n, B in CASES:
            r = uniform_mass(n, B)
            for qb in range(n // B):
                for kb in range(n // B):
                    f.write(f"{n} {B} {qb} {kb} {r[qb][kb].numerator}/{r[qb][kb].denominator}\n")
    with open(os.path.join(HERE, "uniform_support.txt"), "w") as f:
        f.write("# n B tau qb blocks exact_hit   (arg-min support of Section 5.1, eq. "
                "block_working_set, on the uniform masses; exhaustive, exact; no forced blocks)\n")
        for n, B in CASES:
            r = uniform_mass(n, B)
            for tau in TAUS:
                for qb in range(n // B):
                    s = best_support(r[qb], qb, tau)
                    f.write(f"{n} {B} {tau.numerator}/{tau.denominator} {qb} "
                            f"{','.join(str(b) for b in s) if s else '-'} "
                            f"{exact_hit(r[qb], qb, tau)}\n")


if __name__ == "__main__":
    main()
