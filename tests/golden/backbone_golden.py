"""Stored fp64-oracle results of the shared backbone at full size -- test
infrastructure.

The defining statement of group execution (Sec. 5.2) is per tenant: every
tenant receives what its samples would get from a forward run on their own.
At the full-size workloads the oracle needs seconds to minutes per sample, so
this module computes, once and on the CPU, the oracle's result for chosen
samples of *every* tenant and stores it under ``tests/golden/``; the GPU tests
compare against the stored values.

Writing (``python tests/golden/backbone_golden.py 2 3 4 5 6 7``) calls only
``oracle`` (the fp64 per-sample backbone forward and the pooling) and
``workloads`` (the seeded input draws).  Nothing here reads the HIP path.

Stored per chosen sample (``backbone_cfg<N>.npz``, loaded with
``allow_pickle=False``):
  keys [S, 2]       (request, sample) of the sample in the default workload
  lengths [S]       valid rows
  maxabs [S]        max |z| over the sample's valid hidden rows (the scale of
                    the per-sample max-relative bar)
  pooled [S, d]     mean of the valid hidden rows (the MLP heads' feature)
  row_idx [S, R]    rows stored in full: the first, the last and R-2 seeded picks
  rows [S, R, d]    those hidden rows (fp32 copies of the fp64 values)
  dirs [4, d]       four fixed random unit vectors
  proj [sum L, 4]   every valid row's projection onto the four directions (fp32)
  proj_off [S + 1]  first projection row of each sample
  key               sha256 of the drawn inputs the values belong to (backbone
                    spec, every weight, the final gain, the chosen samples'
                    embeddings and lengths); a workload that draws anything
                    else is refused instead of being compared.
"""
from __future__ import annotations

import hashlib
import os
import sys
from typing import Dict, List, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
N_ROWS = 8      # hidden rows stored in full per sample
N_DIRS = 4      # projection directions


def path(cfg: int) -> str:
    return os.path.join(HERE, f"backbone_cfg{cfg}.npz")


def chosen_samples(wl) -> List[Tuple[int, int]]:
    """Per tenant, in tenant order: on the 2B-shaped (18-layer d2048)
    backbones and in groups of eight or more tenants one sample (the
    tenant's first for even tenants, its last for odd ones, so with an even
    tenant count the batch's last sample -- rows in the GEMMs' row-split
    tail -- is included); otherwise the first and the last sample of every
    tenant."""
    big = wl.spec.backbone.d >= 2048 or wl.spec.G >= 8
    out = []
    for g in range(wl.spec.G):
        rows = [(r, s) for r, q in enumerate(wl.requests) if q.tenant == g for s in range(q.n)]
        if big:
            out.append(rows[0] if g % 2 == 0 else rows[-1])
        else:
            out.extend(dict.fromkeys([rows[0], rows[-1]]))
    return out


def input_key(wl, keys) -> str:
    """sha256 over the backbone spec, every backbone weight, the final gain
    and the chosen samples' valid embedding rows and lengths."""
    h = hashlib.sha256()
    h.update(repr(wl.spec.backbone).encode())
    for L in wl.layers:
        for name in sorted(L):
            h.update(name.encode())
            h.update(np.ascontiguousarray(L[name]))
    h.update(np.ascontiguousarray(wl.gf))
    for r, s in keys:
        q = wl.requests[r]
        n = int(q.lengths[s])
        h.update(np.int64([r, s, n]).tobytes())
        h.update(np.ascontiguousarray(q.embeds[s, :n]))
    return h.hexdigest()


def _row_picks(L: int, cfg: int, i: int) -> np.ndarray:
    rng = np.random.default_rng([0x601D, cfg, i])
    picks = [0, L - 1] + [int(x) for x in rng.integers(0, L, N_ROWS - 2)]
    return np.asarray(picks, np.int32)


def make(cfg: int) -> str:
    """Run the fp64 oracle on the chosen samples of workload ``cfg`` and
    store the results."""
    import oracle
    import workloads
    wl = workloads.make_workload(cfg)
    keys = chosen_samples(wl)
    key = input_key(wl, keys)
    res = oracle.step.isolated(wl, samples=keys, heads=False)
    d = wl.spec.backbone.d
    dirs = np.random.default_rng([0xD1125, cfg]).standard_normal((N_DIRS, d))
    dirs /= np.linalg.norm(dirs, axis=1, keepdims=True)
    lengths, maxabs, pooled, row_idx, rows, proj, off = [], [], [], [], [], [], [0]
    for i, k in enumerate(keys):
        z = res["hidden"][k]
        L = z.shape[0]
        lengths.append(L)
        maxabs.append(float(np.max(np.abs(z))))
        pooled.append(res["pooled"][k])
        ri = _row_picks(L, cfg, i)
        row_idx.append(ri)
        rows.append(z[ri].astype(np.float32))
        proj.append((z @ dirs.T).astype(np.float32))
        off.append(off[-1] + L)
    np.savez(path(cfg), keys=np.asarray(keys, np.int32), lengths=np.asarray(lengths, np.int32),
             maxabs=np.asarray(maxabs), pooled=np.stack(pooled), row_idx=np.stack(row_idx),
             rows=np.stack(rows), dirs=dirs, proj=np.concatenate(proj), proj_off=np.asarray(off, np.int64),
             key=np.asarray(key))
    return path(cfg)


def load(cfg: int) -> Dict[str, np.ndarray]:
    with np.load(path(cfg), allow_pickle=False) as f:
        return {k: f[k] for k in f.files}


def compare(wl, gold: Dict[str, np.ndarray], hidden: np.ndarray, cu: np.ndarray,
            pooled: np.ndarray = None) -> Dict[str, float]:
    """Compare a device result with the stored oracle values, sample by sample.

    ``hidden``: the device's hidden rows [T, d] as floats; ``cu``: its
    cu_seqlens; ``pooled`` (optional): its pooled features [N, d] in tenant
    order.  Per chosen sample, relative to that sample's max |z| (the
    per-sample max-relative reading of the 2e-2 bar): the stored rows
    elementwise, every row's four projections, and the pooled feature
    (relative to its own max).  Returns the worst value of each measure and
    the tenant-wise worst, after checking the input key.
    """
    keys = [tuple(int(v) for v in k) for k in gold["keys"]]
    want = str(gold["key"])
    got = input_key(wl, keys)
    if got != want:
        raise AssertionError(f"stored oracle values belong to other inputs (key {want[:12]} != {got[:12]})")
    flat = [(r, s) for r, q in enumerate(wl.requests) for s in range(q.n)]
    index = {k: i for i, k in enumerate(flat)}
    torder = {k: j for j, k in enumerate((r, s) for g in range(wl.spec.G) for r, q in enumerate(wl.requests)
                                         if q.tenant == g for s in range(q.n))}
    tenant_of = {k: wl.requests[k[0]].tenant for k in keys}
    out = {"rows": 0.0, "proj": 0.0, "pooled": 0.0, "samples": len(keys), "tenants": len(set(tenant_of.values()))}
    per_tenant: Dict[int, float] = {}
    for j, k in enumerate(keys):
        i = index[k]
        L = int(gold["lengths"][j])
        if int(cu[i + 1] - cu[i]) < L or int(wl.requests[k[0]].lengths[k[1]]) != L:
            raise AssertionError(f"sample {k}: length mismatch")
        z = np.asarray(hidden[cu[i]: cu[i] + L], np.float64)
        scale = float(gold["maxabs"][j])
        e_rows = float(np.max(np.abs(z[gold["row_idx"][j]] - gold["rows"][j]))) / scale
        p0, p1 = gold["proj_off"][j], gold["proj_off"][j + 1]
        e_proj = float(np.max(np.abs(z @ gold["dirs"].T - gold["proj"][p0:p1]))) / scale
        e = max(e_rows, e_proj)
        out["rows"] = max(out["rows"], e_rows)
        out["proj"] = max(out["proj"], e_proj)
        if pooled is not None:
            p = np.asarray(pooled[torder[k]], np.float64)
            ref = gold["pooled"][j]
            e_pool = float(np.max(np.abs(p - ref)) / np.max(np.abs(ref)))
            out["pooled"] = max(out["pooled"], e_pool)
            e = max(e, e_pool)
        g = tenant_of[k]
        per_tenant[g] = max(per_tenant.get(g, 0.0), e)
    out["per_tenant"] = per_tenant
    out["worst"] = max(per_tenant.values())
    return out


if __name__ == "__main__":
    sys.path.insert(0, ROOT)
    import time
    for a in sys.argv[1:]:
        t0 = time.time()
        p = make(int(a))
        print(f"config {a}: {p} ({os.path.getsize(p) / 1e6:.2f} MB) in {time.time() - t0:.1f} s", flush=True)
