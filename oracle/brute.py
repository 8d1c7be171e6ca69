"""Pure-Python scalar loops of the operator definitions, for tiny shapes.

TEST INFRASTRUCTURE ONLY (see the package docstring).

These are the definitions of ``oracle.ops`` written once more as nested
scalar loops over output elements and reduction indices, with explicit bounds
tests in place of padded copies.  They are slow (use only shapes with at most
a few million multiply-adds) and exist to pin the vectorised float64 versions.
Inputs are nested lists or arrays; outputs are nested Python lists.
"""

import math


def conv2d(x, w, strides=(1, 1), padding=(0, 0, 0, 0), groups=1):
    n_, c_, h_, w_ = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    k_, cg, r_, s_ = len(w), len(w[0]), len(w[0][0]), len(w[0][0][0])
    sh, sw = strides
    pt, pl, pb, pr = padding
    p_ = (h_ + pt + pb - r_) // sh + 1
    q_ = (w_ + pl + pr - s_) // sw + 1
    kg = k_ // groups
    y = [[[[0.0] * q_ for _ in range(p_)] for _ in range(k_)] for _ in range(n_)]
    for n in range(n_):
        for k in range(k_):
            g = k // kg
            for p in range(p_):
                for q in range(q_):
                    acc = 0.0
                    for c in range(cg):
                        ci = g * cg + c
                        for r in range(r_):
                            hi = p * sh - pt + r
                            if hi < 0 or hi >= h_:
                                continue
                            for s in range(s_):
                                wi = q * sw - pl + s
                                if wi < 0 or wi >= w_:
                                    continue
                                acc += float(x[n][ci][hi][wi]) * float(w[k][c][r][s])
                    y[n][k][p][q] = acc
    return y


def dense(x, w):
    return [[sum(float(x[m][k]) * float(w[j][k]) for k in range(len(x[m])))
             for j in range(len(w))] for m in range(len(x))]


def max_pool2d(x, pool_size=(3, 3), strides=(2, 2), padding=(1, 1, 1, 1)):
    n_, c_, h_, w_ = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    r_, s_ = pool_size
    sh, sw = strides
    pt, pl, pb, pr = padding
    p_ = (h_ + pt + pb - r_) // sh + 1
    q_ = (w_ + pl + pr - s_) // sw + 1
    y = [[[[0.0] * q_ for _ in range(p_)] for _ in range(c_)] for _ in range(n_)]
    for n in range(n_):
        for c in range(c_):
            for p in range(p_):
                for q in range(q_):
                    best = -math.inf
                    for r in range(r_):
                        hi = p * sh - pt + r
                        for s in range(s_):
                            wi = q * sw - pl + s
                            if 0 <= hi < h_ and 0 <= wi < w_:
                                best = max(best, float(x[n][c][hi][wi]))
                    y[n][c][p][q] = best
    return y


def global_avg_pool2d(x):
    out = []
    for img in x:
        row = []
        for ch in img:
            tot = 0.0
            cnt = 0
            for line in ch:
                for v in line:
                    tot += float(v)
                    cnt += 1
            row.append(tot / cnt)
        out.append(row)
    return out


def gelu(v):
    return v * 0.5 * math.erfc(-v / math.sqrt(2.0))


def avg_pool2d(x, pool_size=(3, 3), strides=(1, 1), padding=(1, 1, 1, 1), count_include_pad=False):
    n_, c_, h_, w_ = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    r_, s_ = pool_size
    sh, sw = strides
    pt, pl, pb, pr = padding
    p_ = (h_ + pt + pb - r_) // sh + 1
    q_ = (w_ + pl + pr - s_) // sw + 1
    y = [[[[0.0] * q_ for _ in range(p_)] for _ in range(c_)] for _ in range(n_)]
    for n in range(n_):
        for c in range(c_):
            for p in range(p_):
                for q in range(q_):
                    tot, cnt = 0.0, 0
                    for r in range(r_):
                        hi = p * sh - pt + r
                        for s in range(s_):
                            wi = q * sw - pl + s
                            if 0 <= hi < h_ and 0 <= wi < w_:
                                tot += float(x[n][c][hi][wi])
                                cnt += 1
                    y[n][c][p][q] = tot / (r_ * s_ if count_include_pad else cnt)
    return y
