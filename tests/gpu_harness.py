"""Shared helpers of the GPU parity tests: run the library's four calls through
the C ABI, read the documented buffers back, and build the oracle's expected
values in the same order. The oracle and the library never exchange data
except through these comparisons (oracle inputs come from synth only)."""
import sys

import numpy as np
import torch

from oracle import encode, formats, partition, pipeline, rank
from paper_2609_32628_amd import _lib, api
from synth import configs, gen
from fraglayout import mx_section, nv_section, to_frag

TOL_MAX_ABS = 2e-2     # output tolerances of the parity bar
TOL_REL_L2 = 5e-3
NEAR_TIE_REL = 1e-6    # mask mismatches allowed only this close to a threshold score

# A small ragged case: 3 frames of 13x21 tokens (2x3 tiles, edge tiles 40 / 24 / 15 ...).
SMALL = configs.Workload("small-3x13x21-h2-d128", B=2, H=2, d=128, T=3, Hg=13, Wg=21, dtype="bf16",
                         budgets=(10, 30, 100), scope="head", head_scale=True, seed=11)


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def problem_of(w):
    return api.problem(w.B, w.H, w.d, w.T, w.Hg, w.Wg, w.partition)


def inputs(w, heads=None):
    Q, K, V = gen.generate(w, heads)
    return Q, K, V


def to_device(X, w):
    t = torch.from_numpy(np.ascontiguousarray(X))
    return t.to(torch.bfloat16 if w.dtype == "bf16" else torch.float32).cuda()


SECTION_NAMES = ["Q4", "K4", "V4", "Q8", "K8", "V8", "dQ", "dK", "dV", "g", "Q16", "K16", "V16",
                 "Q4mx", "K4mx", "V4mx"]


def section_specs(p, R):
    """(dtype, per-head shape) of each ops section, in da2_ops_offsets order."""
    d = p.d
    mx = (d // 32 + 1) * 1024
    return [(np.uint8, (R, 36 * d)), (np.uint8, (R, 36 * d)), (np.uint8, (R, 36 * d)),
            (np.int8, (R, 64 * d)), (np.int8, (R, 64 * d)), (np.uint8, (R, 64 * d)),
            (np.float32, (R,)), (np.float32, (R,)), (np.float32, (d,)), (np.float32, (4,)),
            (np.float16, (R, 64 * d)), (np.float16, (R, 64 * d)), (np.float16, (R, 64 * d)),
            (np.uint8, (R, mx)), (np.uint8, (R, mx)), (np.uint8, (R, mx))]


def ops_tag(fmt4, with16):
    """The encoding tag prep writes into word 3 of each head's g entry."""
    return (_lib.TAG_MARKER | (_lib.DA2_OPS_LAYOUT_VERSION << 8) | (0x10 if with16 else 0)
            | {"nvfp4": 0, "mxfp4": 1}[fmt4])


def sections(buf, p):
    """Encoded operands of the ops buffer as numpy arrays [BH, R, ...] (the
    sections the buffer holds for its fmt4 / with16)."""
    off = api.da2_ops_offsets(p, buf.fmt4, buf.with16)
    raw = buf.ops.cpu().numpy()
    BH, R = p.B * p.H, buf.sizes["R"]
    out = {}
    for i, (name, (dt, shape)) in enumerate(zip(SECTION_NAMES, section_specs(p, R))):
        if off[i] < 0:
            continue
        nbytes = BH * int(np.prod(shape)) * np.dtype(dt).itemsize
        out[name] = raw[off[i]:off[i] + nbytes].view(dt).reshape((BH,) + shape)
    return out


def lists_of(buf, p):
    lo = api.da2_lists_offsets(p)
    raw = buf.lists.cpu().numpy()
    BH, R = p.B * p.H, buf.sizes["R"]
    keys = raw[lo[0]:lo[0] + 2 * BH * R * R].view(np.uint16).reshape(BH * R, R)
    counts = raw[lo[1]:lo[1] + 16 * BH * R].view(np.int32).reshape(BH * R, 4)
    order = raw[lo[2]:lo[2] + 4 * BH * R].view(np.int32)
    return keys, counts, order


def write_lists(buf, p, cls_all):
    """Oracle class maps [BH, R, R] -> the lists section (identity work order)."""
    lo = api.da2_lists_offsets(p)
    BH, R = cls_all.shape[0], cls_all.shape[1]
    keys = np.zeros((BH * R, R), np.uint16)
    counts = np.zeros((BH * R, 4), np.int32)
    for i, row in enumerate(cls_all.reshape(BH * R, R)):
        l4, l8, l16 = rank.key_lists_all(row)
        seg = np.concatenate([l4, l8, l16])
        keys[i, :seg.size] = seg
        counts[i] = (l4.size, l8.size, l16.size, 0)
    raw = buf.lists.cpu().numpy()
    raw[lo[0]:lo[0] + keys.nbytes] = keys.view(np.uint8).reshape(-1)
    raw[lo[1]:lo[1] + counts.nbytes] = counts.view(np.uint8).reshape(-1)
    order = np.arange(BH * R, dtype=np.int32)
    raw[lo[2]:lo[2] + order.nbytes] = order.view(np.uint8)
    buf.lists.copy_(torch.from_numpy(raw))


def expected_mx_sections(enc_mx):
    """Oracle MXFP4 encodings of one head as the bytes of sections 13..15."""
    return {name + "4mx": mx_section(name, formats.e2m1_code(enc_mx["e" + name]), enc_mx["k" + name])
            for name in ("Q", "K", "V")}


def expected_sections(enc, enc_mx=None, fmt4="nvfp4", with16=True):
    """Oracle encodings of one head in the ops-buffer order (the MXFP4
    sections only when ``enc_mx`` is given; the g tag for fmt4 / with16)."""
    mx = {} if enc_mx is None else expected_mx_sections(enc_mx)
    tag = np.array([ops_tag(fmt4, with16)], np.uint32).view(np.float32)[0]
    return {
        **mx,
        "Q4": nv_section("Q", formats.e2m1_code(enc["eQ"]), formats.e4m3_code(enc["sQ"])),
        "K4": nv_section("K", formats.e2m1_code(enc["eK"]), formats.e4m3_code(enc["sK"])),
        "V4": nv_section("V", formats.e2m1_code(enc["eV"]), formats.e4m3_code(enc["sV"])),
        "Q8": to_frag("Q8", enc["q8"]), "K8": to_frag("K8", enc["k8"]),
        "V8": to_frag("V8", formats.e4m3_code(enc["v8"])),
        "dQ": enc["dQ"], "dK": enc["dK"], "dV": enc["dV"],
        "g": np.array([enc["gQ"], enc["gK"], enc["gV"], tag], np.float32),
        "Q16": to_frag("Q16", enc["q16"].astype(np.float64)), "K16": to_frag("K16", enc["k16"].astype(np.float64)),
        "V16": to_frag("V16", enc["v16"].astype(np.float64)),
    }


def write_ops(buf, p, encs, encs_mx=None):
    """Oracle encodings of every head -> the sections the ops buffer holds
    (stage injection): the 4-bit encoding of the buffer's fmt4 (MXFP4 from
    ``encs_mx``), the 16-bit sections when the buffer has them, and the g tag."""
    off = api.da2_ops_offsets(p, buf.fmt4, buf.with16)
    raw = buf.ops.cpu().numpy()
    exp = [expected_sections(e, None if encs_mx is None else encs_mx[i], buf.fmt4, buf.with16)
           for i, e in enumerate(encs)]
    for i, name in enumerate(SECTION_NAMES):
        if off[i] < 0:
            continue
        arr = np.stack([x[name] for x in exp])
        b = np.ascontiguousarray(arr).view(np.uint8).reshape(-1)
        raw[off[i]:off[i] + b.size] = b
    buf.ops.copy_(torch.from_numpy(raw))


def compare_outputs(O_gpu, O_ref, label, diag=None):
    """Parity bar on the rows where O_ref is defined (not NaN). When the bar
    fails and ``diag`` is given, diag(row indices of O_ref's leading axes)
    reports the worst rows before the assertion."""
    rows = ~np.isnan(O_ref).any(axis=-1)
    a, b = O_gpu[rows].astype(np.float64), O_ref[rows]
    err = np.abs(a - b)
    max_abs = float(err.max()) if err.size else 0.0
    rel = float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))
    log(f"[{label}] rows={int(rows.sum())} max_abs={max_abs:.3e} rel_l2={rel:.3e}")
    if diag is not None and (max_abs > TOL_MAX_ABS or rel > TOL_REL_L2):
        row_err = np.where(rows, np.nanmax(np.abs(O_gpu.astype(np.float64) - np.nan_to_num(O_ref)), axis=-1), -1.0)
        worst = np.argsort(row_err, axis=None)[::-1][:3]
        diag([np.unravel_index(i, row_err.shape) for i in worst])
    assert max_abs <= TOL_MAX_ABS, (label, max_abs)
    assert rel <= TOL_REL_L2, (label, rel)
    return max_abs, rel


def boundary_distance(x, table):
    """Relative distance of each |x| to the nearest rounding boundary (the
    midpoint of two neighbouring magnitudes) of a format with value table."""
    t = np.unique(np.abs(table[np.isfinite(table)]))
    mids = (t[1:] + t[:-1]) / 2
    ax = np.abs(np.asarray(x, np.float64))
    i = np.searchsorted(mids, ax)
    lo = mids[np.clip(i - 1, 0, mids.size - 1)]
    hi = mids[np.clip(i, 0, mids.size - 1)]
    return np.minimum(np.abs(ax - lo), np.abs(ax - hi)) / np.maximum(ax, 1e-300)


def flip_report(ops, a, lists, u, label=""):
    """For query u of region a: the weights whose quantizer input lies closest
    to a rounding boundary (the NVFP4 2688 P/sigma_P on E2M1, the INT8 path's
    amplified P on E4M3). A GPU/oracle difference with a distance near float32
    rounding (about 1e-7) is a rounding flip, not a defect."""
    from oracle import attention as oatt
    _, parts = oatt.attend(ops, a, *lists, return_parts=True)
    Pt = parts["Pt"][u]                                       # [nb, 64]
    n4, n8 = len(lists[0]), len(lists[1])
    found = []
    if n4:
        g = Pt[:n4].reshape(n4, 4, 16)
        sigma = formats.e4m3(448.0 * g.max(axis=-1))
        y = np.where(sigma[..., None] > 0, oatt.FP4_P_SCALE * g / np.where(sigma > 0, sigma, 1.0)[..., None], 0.0)
        dist = boundary_distance(y, formats.E2M1_VALUES).reshape(n4, 64)
        found += [(float(dist[j, v]), "nvfp4", int(lists[0][j]), v) for j, v in zip(*np.nonzero(Pt[:n4] > 0))]
    if n8:
        y = oatt.AMP * Pt[n4:n4 + n8]
        dist = boundary_distance(y, formats.e4m3_decode(np.arange(256)))
        found += [(float(dist[j, v]), "int8", int(lists[1][j]), v) for j, v in zip(*np.nonzero(Pt[n4:n4 + n8] > 0))]
    found.sort()
    log(f"  flip report {label} region {a} query {u}: nearest boundaries " +
        ", ".join(f"{p}:block {b} slot {v} rel {dd:.1e}" for dd, p, b, v in found[:6]))


def mask_mismatches(cls_gpu, cls_ref, A_ref, quotas, scope):
    """Count class mismatches; every one must be a near-tie at a threshold
    (the score at cumulative rank T16, T16+T8 or T16+T8+T4) it crossed."""
    bad = np.nonzero(cls_gpu != cls_ref)
    if bad[0].size == 0:
        return 0
    T16, T8, T4 = quotas
    cuts = (T16, T16 + T8, T16 + T8 + T4)
    R = A_ref.shape[0]
    if scope == "head":
        flat = A_ref.reshape(-1).astype(np.float64)
        order = np.lexsort((np.arange(flat.size), -flat))
        thetas = [flat[order[k - 1]] for k in cuts if k > 0]
        for a, b in zip(*bad):
            s = float(A_ref[a, b])
            assert min(abs(s - t) / abs(t) for t in thetas) <= NEAR_TIE_REL, (a, b, s, thetas)
    else:
        for a, b in zip(*bad):
            row = A_ref[a].astype(np.float64)
            order = np.lexsort((np.arange(R), -row))
            thetas = [row[order[k - 1]] for k in cuts if k > 0]
            s = float(A_ref[a, b])
            assert min(abs(s - t) / abs(t) for t in thetas) <= NEAR_TIE_REL, (a, b, s, thetas)
    return bad[0].size
