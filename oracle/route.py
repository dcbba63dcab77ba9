"""Hybrid execution routing and in-GPU compaction layout (oracle), Sec. 3.4-3.5.

Static micro-buckets B = {8, 16, 32, ..., N_max} (Sec. 3.4); the batch-level
boundary max_b L*_b mapped to its bucket is the "naive pad" policy.  For a
sequence group G padded to bucket B_G the padding waste ratio is
    rho = 1 - sum_{i in G} L*_i / (|G| * B_G).
Three paths: Static-Graph when rho <= tau_pad, Bucket-Varlen-Graph when
rho > tau_pad, Eager for isolated stragglers (|G| = 1) or ultra-short groups.

Readings where the paper is silent or inconsistent:
  * coarse clustering: class k(L) = ceil(log_4 max(L, 8)), one group per class
    present, groups numbered in ascending class order, members in (L*, index)
    order;
  * the eager rule "B_G <= 4" cannot fire with buckets that start at 8, so it
    is read as max_{i in G} L*_i <= 4 (or |G| = 1);
  * the bucket set is capped by the longest window N_max of the batch;
  * compaction keeps batch order: sequence b occupies rows
    [cu_dst[b], cu_dst[b+1]) = its prefix, its first L*_b window rows, then zero
    pad rows up to its allocation (B_G on the static path, L*_b otherwise);
    seqused[b] = prefix + L*_b marks where the pad starts, so pad rows are
    masked as keys (the attention-mask rewrite);
  * the packed capacity is the total row count rounded up to a granule (the
    "predefined 1-D graph shape"), the extra rows zero.
"""
from dataclasses import dataclass, field
from fractions import Fraction
from typing import List

import numpy as np

PATH_STATIC, PATH_VARLEN, PATH_EAGER = 0, 1, 2
POLICY_HYBRID, POLICY_NAIVE_PAD, POLICY_VARLEN_ONLY = 0, 1, 2


def bucket_set(n_max):
    out = []
    b = 8
    while b < n_max:
        out.append(b)
        b *= 2
    out.append(int(n_max))
    return out


def bucket_of(length, n_max):
    for b in bucket_set(n_max):
        if b >= length:
            return b
    raise ValueError("length exceeds the largest bucket")


def padding_waste_ratio(lengths, bucket):
    lengths = [int(l) for l in lengths]
    return Fraction(1) - Fraction(sum(lengths), len(lengths) * int(bucket))


def coarse_class(length):
    m = max(int(length), 8)
    k = 0
    while 4 ** k < m:
        k += 1
    return k


@dataclass
class RouteResult:
    path: np.ndarray      # [B] PATH_*
    group: np.ndarray     # [B] group id
    alloc: np.ndarray     # [B] window rows allocated (bucket on the static path)
    groups: List[dict] = field(default_factory=list)


def route_batch(keep_len, win_len, policy=POLICY_HYBRID, tau_pad=Fraction(1, 5)):
    keep = [int(k) for k in keep_len]
    B = len(keep)
    path = np.zeros(B, np.int64)
    group = np.zeros(B, np.int64)
    alloc = np.zeros(B, np.int64)
    groups = []
    if B == 0:
        return RouteResult(path, group, alloc, groups)
    n_max = int(max(int(n) for n in win_len))
    order = sorted(range(B), key=lambda i: (keep[i], i))
    if policy == POLICY_NAIVE_PAD:
        bg = bucket_of(max(keep), n_max)
        for i in order:
            path[i], group[i], alloc[i] = PATH_STATIC, 0, bg
        groups.append({"members": order, "bucket": bg,
                       "pwr": padding_waste_ratio(keep, bg), "path": PATH_STATIC})
        return RouteResult(path, group, alloc, groups)
    if policy == POLICY_VARLEN_ONLY:
        for i in order:
            path[i], group[i], alloc[i] = PATH_VARLEN, 0, keep[i]
        groups.append({"members": order, "bucket": None, "pwr": None, "path": PATH_VARLEN})
        return RouteResult(path, group, alloc, groups)
    if policy != POLICY_HYBRID:
        raise ValueError("unknown policy")
    classes = sorted({coarse_class(keep[i]) for i in order})
    for gid, k in enumerate(classes):
        members = [i for i in order if coarse_class(keep[i]) == k]
        lens = [keep[i] for i in members]
        bg = bucket_of(max(lens), n_max)
        rho = padding_waste_ratio(lens, bg)
        if len(members) == 1 or max(lens) <= 4:
            p = PATH_EAGER
        elif rho <= Fraction(tau_pad):
            p = PATH_STATIC
        else:
            p = PATH_VARLEN
        for i in members:
            path[i], group[i] = p, gid
            alloc[i] = bg if p == PATH_STATIC else keep[i]
        groups.append({"members": members, "bucket": bg, "pwr": rho, "path": p})
    return RouteResult(path, group, alloc, groups)


def repack_rows(src, cu_src, win_off, keep_len, alloc, granule=1):
    """Compaction: gather each sequence's prefix and kept window rows.

    Returns (dst [capacity, d], cu_dst [B+1], seqused [B], capacity).
    """
    src = np.asarray(src)
    cu_src = np.asarray(cu_src, np.int64)
    B = len(cu_src) - 1
    lens = [int(win_off[b]) + int(alloc[b]) for b in range(B)]
    cu_dst = np.zeros(B + 1, np.int64)
    for b in range(B):
        cu_dst[b + 1] = cu_dst[b] + lens[b]
    total = int(cu_dst[B])
    g = max(int(granule), 1)
    capacity = ((total + g - 1) // g) * g
    dst = np.zeros((capacity,) + src.shape[1:], src.dtype)
    seqused = np.zeros(B, np.int64)
    for b in range(B):
        n_keep = int(win_off[b]) + int(keep_len[b])
        s0 = int(cu_src[b])
        d0 = int(cu_dst[b])
        dst[d0:d0 + n_keep] = src[s0:s0 + n_keep]
        seqused[b] = n_keep
    return dst, cu_dst, seqused, capacity
