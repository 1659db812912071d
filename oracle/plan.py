"""Pack plan of a group of requests -- oracle (test infrastructure only).

App. A.3: requests are examined in arrival order; canonicalization and
padding produce one physical encoder batch together with the slices that
later partition the shared features back to their requests.  Sec. 4.3:
the canonical ``VLAFeature`` shape is where concatenation happens.

Readings (the paper fixes no tensor layout):
  * physical order = request arrival order, samples in order inside a
    request (FIFO, App. A.3);
  * a sample occupies ``roundup(len, align)`` consecutive rows; the rows
    past ``len`` are alignment padding (sample -1, position -1);
  * tenant order for the heads is a stable sort of samples by tenant slot
    (ties keep arrival order);
  * a tenant in the table with no sample, a length < 1 or > max_len, or a
    schema signature / model width that differs from the group's, is an
    error (compatibility is decided at the shared-prefix boundary,
    App. A.3, not by tenant identity).

Everything is written with plain Python loops on purpose.
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np


class PlanError(ValueError):
    pass


class Incompatible(PlanError):
    pass


def pack_plan(req_tenant: Sequence[int], req_lengths: Sequence[Sequence[int]],
              req_max_len: Sequence[int], G: int, align: int = 1,
              tenant_sig: Sequence[int] = None, tenant_d: Sequence[int] = None,
              d: int = None) -> Dict[str, np.ndarray]:
    """Index maps of the physical batch.

    Returns int32 arrays
      seqlens[N], cu_seqlens[N+1], sample_request[N], sample_local[N],
      sample_tenant[N], tenant_sample_off[G+1], tenant_perm[N],
      sample_tenant_rank[N], token_sample[T], token_pos[T]
    plus ints N, T.
    """
    if align < 1:
        raise PlanError("align must be >= 1")
    R = len(req_tenant)
    if R < 1 or G < 1:
        raise PlanError("need at least one request and one tenant")
    if tenant_sig is not None:
        for g in range(G):
            if tenant_sig[g] != tenant_sig[0]:
                raise Incompatible(f"tenant {g} has a different shared-prefix signature")
    if tenant_d is not None and d is not None:
        for g in range(G):
            if tenant_d[g] != d:
                raise Incompatible(f"tenant {g} expects width {tenant_d[g]}, backbone has {d}")

    seqlens: List[int] = []
    s_req: List[int] = []
    s_loc: List[int] = []
    s_ten: List[int] = []
    for r in range(R):
        g = int(req_tenant[r])
        if g < 0 or g >= G:
            raise PlanError(f"request {r} names tenant {g} outside the table")
        if len(req_lengths[r]) < 1:
            raise PlanError(f"request {r} has no samples")
        for s in range(len(req_lengths[r])):
            L = int(req_lengths[r][s])
            if L < 1 or L > int(req_max_len[r]):
                raise PlanError(f"request {r} sample {s}: length {L} outside [1, {req_max_len[r]}]")
            seqlens.append(L)
            s_req.append(r)
            s_loc.append(s)
            s_ten.append(g)
    N = len(seqlens)

    cu = [0]
    for i in range(N):
        rows = ((seqlens[i] + align - 1) // align) * align
        cu.append(cu[-1] + rows)
    T = cu[-1]
    if T >= 2 ** 31:
        raise PlanError("packed batch overflows int32 row indices")

    token_sample = [-1] * T
    token_pos = [-1] * T
    for i in range(N):
        for j in range(seqlens[i]):
            token_sample[cu[i] + j] = i
            token_pos[cu[i] + j] = j

    counts = [0] * G
    for i in range(N):
        counts[s_ten[i]] += 1
    for g in range(G):
        if counts[g] == 0:
            raise PlanError(f"tenant {g} has no samples in this group")
    off = [0]
    for g in range(G):
        off.append(off[-1] + counts[g])

    perm: List[int] = []
    for g in range(G):
        for i in range(N):
            if s_ten[i] == g:
                perm.append(i)
    rank = [0] * N
    for k in range(N):
        rank[perm[k]] = k

    i32 = lambda v: np.array(v, dtype=np.int32)  # noqa: E731
    return {
        "N": N, "T": T,
        "seqlens": i32(seqlens), "cu_seqlens": i32(cu),
        "sample_request": i32(s_req), "sample_local": i32(s_loc), "sample_tenant": i32(s_ten),
        "tenant_sample_off": i32(off), "tenant_perm": i32(perm), "sample_tenant_rank": i32(rank),
        "token_sample": i32(token_sample), "token_pos": i32(token_pos),
    }


def pack_tokens(plan: Dict[str, np.ndarray], req_embeds: Sequence[np.ndarray]) -> np.ndarray:
    """Physical batch rows (any dtype; bf16 bit patterns in practice).

    Row t holds request r's sample s row j for the (r, s, j) that the plan
    maps to t; alignment rows are zero.
    """
    d = req_embeds[0].shape[-1]
    out = np.zeros((plan["T"], d), dtype=req_embeds[0].dtype)
    for t in range(plan["T"]):
        i = int(plan["token_sample"][t])
        if i < 0:
            continue
        r = int(plan["sample_request"][i])
        s = int(plan["sample_local"][i])
        j = int(plan["token_pos"][t])
        out[t] = req_embeds[r][s, j]
    return out


def unpack_tokens(plan: Dict[str, np.ndarray], rows: np.ndarray,
                  req_shapes: Sequence[tuple]) -> List[np.ndarray]:
    """Inverse of ``pack_tokens``: per-request [n, max_len, width] buffers,
    rows at padding positions zero."""
    outs = [np.zeros(shape, dtype=rows.dtype) for shape in req_shapes]
    for t in range(plan["T"]):
        i = int(plan["token_sample"][t])
        if i < 0:
            continue
        r = int(plan["sample_request"][i])
        s = int(plan["sample_local"][i])
        outs[r][s, int(plan["token_pos"][t])] = rows[t]
    return outs
