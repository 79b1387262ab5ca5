"""Readers for the text fixtures under tests/golden (no MixFP4 arithmetic)."""
import os
from fractions import Fraction

import numpy as np

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _lines(name):
    with open(os.path.join(HERE, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                yield line


def table1():
    codes, fields, books = {}, {}, {}
    for line in _lines("table1_fp4_formats.txt"):
        parts = line.split()
        if parts[1] == "code":
            codes[(parts[0], int(parts[2], 2))] = Fraction(parts[3])
        elif parts[1] == "codebook":
            books[parts[0]] = [Fraction(v) for v in parts[2].split(",")]
        else:
            fields[(parts[0], parts[1])] = Fraction(parts[2])
    return codes, fields, books


def handworked_blocks():
    out = []
    for line in _lines("handworked_blocks.txt"):
        vals, sig, err, t, sb, cb = [p.strip() for p in line.split("|")]
        block = np.zeros(16, dtype=np.float32)
        v = [float(x) for x in vals.split()]
        block[:len(v)] = v
        out.append(dict(
            block=block,
            sigma=tuple(Fraction(s) for s in sig.split()),
            err=tuple(Fraction(e) for e in err.split()),
            t=int(t), scale=int(sb, 16),
            codes=bytes(int(c, 16) for c in cb.split())))
    return out


def handworked_gemm():
    d = {}
    for line in _lines("handworked_gemm.txt"):
        k, *v = line.split()
        d[k] = [float(x) for x in v]
    return d


def philox_kat():
    out = []
    for line in _lines("philox4x32_kat.txt"):
        rounds, ctr, key, words = [p.strip() for p in line.split("|")]
        out.append(dict(rounds=int(rounds),
                        counter=[int(v, 16) for v in ctr.split()],
                        key=[int(v, 16) for v in key.split()],
                        out=[int(v, 16) for v in words.split()]))
    return out


def sr_handworked():
    out = []
    for line in _lines("sr_handworked.txt"):
        grid, y, u, code, _ = [p.strip() for p in line.split("|")]
        out.append(dict(grid=grid, y=float(Fraction(y)), u=int(u), code=int(code)))
    return out
