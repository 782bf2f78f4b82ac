"""GPU rotation matrices (fp32 covariance and cyclic Jacobi on the GPU,
mosaic_compute_rotations) against the rotation oracle (fp64 covariance,
numpy eigh).  Eigenvectors of close eigenvalues are not unique, so the checks
are the properties that define the result: orthonormal rows, the rotated
covariance R C R^T diagonal (off-diagonal energy) with the oracle's
eigenvalues on its diagonal in descending order, the sign rule, the
eigenvectors themselves where a wide eigenvalue gap isolates them, window
repetition past the last token and the identity for an empty sequence.

Tolerances (relative to the largest eigenvalue): the covariance accumulates
exact 16-bit products in fp32 over 4096-token slices, then the
Jacobi rotations accumulate fp32 rounding over a few thousand steps; 5e-5 of
the largest eigenvalue bounds both with margin, and an eigenvector whose gap
to its neighbours is g (relative) moves by about that error over g.
"""
import numpy as np
import pytest
import torch

import paper_2607_00760_amd as M
from oracle import rotation as RO
from workloads import gen

pytestmark = pytest.mark.gpu

D = 128
TOL = 5e-5
SEG_T = 64

CASES = {
    "outliers_fp16": gen.spec("c1", ctx=(2500, 700, 0), hkv=2, rot_window=1024),
    "gauss_bf16": gen.spec("c3", ctx=(1500, 64), hkv=2, kind="gauss", rot_window=1024),
    "student_bf16": gen.spec("c5", ctx=(3000, 100), hkv=2, rot_window=2048, appends=0),
    # one window of 65536 tokens (16 covariance slices) and a short second one
    "long_window": gen.spec("c3", ctx=(70000,), hkv=1, kind="gauss"),
}


def _check_window(Rg, eg, Ro, eo, X, where):
    lam = max(float(eo[0]), 1e-30)
    assert np.abs(Rg @ Rg.T - np.eye(D)).max() <= 3e-5, f"{where}: rows not orthonormal"
    Cm = X.T @ X
    Mr = Rg @ Cm @ Rg.T
    dg = np.diag(Mr)
    assert np.abs(dg - eo).max() <= TOL * lam, f"{where}: Rayleigh quotients vs oracle eigenvalues"
    assert np.abs(Mr - np.diag(dg)).max() <= TOL * lam, f"{where}: rotated covariance not diagonal"
    assert np.abs(eg - eo).max() <= TOL * lam, f"{where}: eigenvalues"
    assert np.all(np.diff(eg) <= 0), f"{where}: eigenvalues not descending"
    top = np.argmax(np.abs(Rg), axis=1)
    assert np.all(Rg[np.arange(D), top] > 0), f"{where}: sign rule"
    gaps = np.abs(np.diff(eo))
    gap = np.minimum(np.concatenate([[np.inf], gaps]), np.concatenate([gaps, [np.inf]])) / lam
    srt = np.sort(np.abs(Ro), axis=1)
    clear_sign = (srt[:, -1] - srt[:, -2]) > 1e-3                  # largest component not nearly tied
    iso = np.nonzero((gap > 1e-2) & clear_sign)[0]
    for i in iso:
        err = np.abs(Rg[i] - Ro[i]).max()
        assert err <= 2 * TOL / gap[i] + 1e-5, f"{where}: eigenvector {i} (gap {gap[i]:.3g}) off by {err:.3g}"
    return len(iso)


@pytest.mark.parametrize("name", list(CASES))
def test_rotations_match_oracle(name):
    spec = CASES[name]
    print(f"[rotation] {name} ctx={spec.ctx} W={spec.rot_window} {spec.dtype}", flush=True)
    cap = spec.max_ctx
    lay = gen.make_layer(spec, 0, capacity=cap)
    params = M.Params(num_kv_heads=spec.hkv, group_size=spec.group, dtype=spec.dtype, rot_window=spec.rot_window)
    k, v = lay["k"].cuda(), lay["v"].cuda()
    rk, rv, ek, ev = M.compute_rotations(params, k, v, spec.ctx, cap, evals=True)
    torch.cuda.synchronize()
    out = {"k": (rk.double().cpu().numpy(), ek.double().cpu().numpy()),
           "v": (rv.double().cpu().numpy(), ev.double().cpu().numpy())}
    nw = -(-cap // spec.rot_window)
    n_iso = 0
    for b in range(spec.num_seqs):
        L = spec.ctx[b]
        for h in range(spec.hkv):
            for which in ("k", "v"):
                x = lay[which][b, h].double().numpy()          # 16-bit inputs, exact in fp64
                Ro, eo = RO.rotations(x, L, spec.rot_window, nw)
                Rg, eg = out[which][0][b, h], out[which][1][b, h]
                nwt = -(-L // spec.rot_window)
                if nwt == 0:
                    for w in range(nw):
                        assert np.array_equal(Rg[w], np.eye(D)) and not eg[w].any(), f"{name}: empty sequence"
                    continue
                for w in range(nw):
                    if w >= nwt:
                        assert np.array_equal(Rg[w], Rg[nwt - 1]), f"{name}: window {w} repeats {nwt - 1}"
                        continue
                    a, e = w * spec.rot_window, min((w + 1) * spec.rot_window, L)
                    n_iso += _check_window(Rg[w], eg[w], Ro[w], eo[w], x[a:e], f"{name} seq {b} head {h} {which} w{w}")
    print(f"[rotation] {name}: {n_iso} isolated eigenvectors compared", flush=True)


def test_rotations_feed_compress():
    """The GPU rotations, handed to mosaic_compress on the device, are used as
    R (rows = eigenvectors): every kept K value of the first segment of every
    pair is x . R^T (fp64 from the same fp32 R) rounded to the cache dtype,
    and the kept channels are the r largest |y| (ties within the fp32
    rounding of y aside).  This checks the hand-over only: compression with a
    given R is pinned against the oracle by the parity tests, and R itself
    against the oracle's eigendecomposition above."""
    spec = gen.spec("c2", ctx=(1500, 700), hkv=2, rot_window=1024)
    cap = spec.max_ctx
    lay = gen.make_layer(spec, 0, capacity=cap)
    params = M.Params(num_kv_heads=spec.hkv, group_size=1, dtype=spec.dtype, rot_window=spec.rot_window,
                      force_default=True)
    k, v = lay["k"].cuda(), lay["v"].cuda()
    rk, rv = M.compute_rotations(params, k, v, spec.ctx, cap)
    c = M.MosaicCache(params, spec.num_seqs, cap, rotated=True)
    c.compress(k, v, lay["ctx_lens"], rk, rv)
    torch.cuda.synchronize()
    R = rk.double().cpu().numpy()
    fdt = {"bf16": torch.bfloat16, "fp16": torch.float16}[spec.dtype]
    for pi in range(spec.num_seqs * spec.hkv):
        b, h = divmod(pi, spec.hkv)
        d = c.region("desc", pi, 16).cpu().numpy()
        tok_off = int(d[:4].view(np.uint32)[0])
        r, l2g, l2b = int(d[12]), int(d[13]), int(d[14])
        assert l2g == 0, "default strategy has one channel per group"
        B, bmb = 1 << l2b, 16
        x = lay["k"][b, h, :SEG_T].double().numpy()
        y = x @ R[b, h, 0].T
        arena = c.region("token", pi, tok_off + (SEG_T // B) * B * 2 * (bmb + 2 * r)).cpu().numpy()[tok_off:]
        for t in range(SEG_T):
            blk = arena[(t // B) * B * 2 * (bmb + 2 * r):]
            j = t % B
            bm = np.unpackbits(blk[j * bmb:(j + 1) * bmb], bitorder="little").astype(bool)
            vals = blk[B * bmb + j * 2 * r: B * bmb + (j + 1) * 2 * r].view(np.uint16)
            got = torch.from_numpy(vals.view(np.int16).copy()).view(fdt).double().numpy()
            ch = np.nonzero(bm)[0]
            assert ch.size == r, f"pair {pi} token {t}: {ch.size} kept"
            ay = np.abs(y[t])
            # one rounding to 16 bits (at most 2^-8 relative for bf16) after the fp32 sums
            tol_v = np.abs(y[t, ch]) * 2.0 ** -7 + 1e-5 * ay.max()
            assert np.all(np.abs(got - y[t, ch]) <= tol_v), f"pair {pi} token {t}: kept values are not x . R^T"
            thr = np.sort(ay)[-r]
            tol = 1e-5 * ay.max()
            assert np.all(ay[ch] >= thr - tol) and np.all(ay[~bm] <= thr + tol), \
                f"pair {pi} token {t}: kept channels are not the r largest"


@pytest.mark.parametrize("name,keep", [("c2_fp16", 32), ("c3_bf16_r16", 16)])
def test_reorder_matches_oracle(name, keep):
    """mosaic_reorder_rotations against the oracle's selection-pattern reorder
    on the same fp32 matrices (the oracle's eigenbases): the reordered
    matrices are identical bit for bit (the counts are integers over the
    compressor's exact fp32 chain), including windows without tokens and an
    empty sequence."""
    spec = (gen.spec("c2", ctx=(1500, 700, 0), hkv=2, rot_window=1024) if name == "c2_fp16"
            else gen.spec("c3", ctx=(2100, 64), hkv=2, kind="gauss", rot_window=1024))
    print(f"[reorder] {name} ctx={spec.ctx} r={keep}", flush=True)
    cap = spec.max_ctx + 1024                                 # one window past the longest context
    lay = gen.make_layer(spec, 0, capacity=cap)
    W, nw = spec.rot_window, -(-cap // spec.rot_window)
    R = {}
    for which in ("k", "v"):
        R[which] = np.zeros((spec.num_seqs, spec.hkv, nw, D, D), np.float32)
        for b in range(spec.num_seqs):
            for h in range(spec.hkv):
                R[which][b, h] = RO.rotations(lay[which][b, h].double().numpy(), spec.ctx[b], W, nw)[0]
    params = M.Params(num_kv_heads=spec.hkv, group_size=spec.group, dtype=spec.dtype, rot_window=W,
                      default=(keep, 1, 8))
    rk, rv = torch.from_numpy(R["k"]).cuda(), torch.from_numpy(R["v"]).cuda()
    M.reorder_rotations(params, lay["k"].cuda(), lay["v"].cuda(), spec.ctx, cap, rk, rv)
    torch.cuda.synchronize()
    got = {"k": rk.cpu().numpy(), "v": rv.cpu().numpy()}
    moved = 0
    for b in range(spec.num_seqs):
        L = spec.ctx[b]
        for h in range(spec.hkv):
            for which in ("k", "v"):
                x = lay[which][b, h].float().numpy()
                want, orders = RO.reorder_rotations(x, L, W, R[which][b, h], keep)
                assert np.array_equal(got[which][b, h], want), f"{name} seq {b} head {h} {which}"
                moved += int((orders != np.arange(D)).any(axis=1).sum())
    print(f"[reorder] {name}: {moved} windows reordered", flush=True)
    assert moved > 0


def test_coselection_reorder_moves_the_ratio():
    """Channels that are always selected together (features of four channels,
    equal selection counts) under given rotations that scatter them: the
    strategy search keeps single channels, (16, 1).  mosaic_reorder_rotations
    (bit-exact against the oracle's co-selection order) groups each feature,
    the search then takes (16, 4) and the compressed cache shrinks; both
    compressions are byte-exact against the oracle."""
    from _parity import assert_state_equal, bits
    from oracle import oracle as O
    ns, hkv, L = 2, 2, 2048
    k = torch.empty((ns, hkv, L, D), dtype=torch.float16)
    v = torch.empty_like(k)
    rk = torch.empty((ns, hkv, 1, D, D))
    rv = torch.empty_like(rk)
    for b in range(ns):
        for h in range(hkv):
            k[b, h] = gen.feature_tokens(("k", b, h), L).half()
            v[b, h] = gen.feature_tokens(("v", b, h), L).half()
            rk[b, h, 0] = gen.signed_permutation(("k", b, h))
            rv[b, h, 0] = gen.signed_permutation(("v", b, h))
    params = M.Params(num_kv_heads=hkv, group_size=4, dtype="fp16", rot_window=L, default=(16, 4, 8))
    op = O.Params(group=4, dtype="fp16", rot_window=L, default=(16, 4, 8))
    rk2, rv2 = rk.clone().cuda(), rv.clone().cuda()
    M.reorder_rotations(params, k.cuda(), v.cuda(), [L] * ns, L, rk2, rv2)
    torch.cuda.synchronize()
    for b in range(ns):
        for h in range(hkv):
            for R0, Rg, x in ((rk, rk2, k), (rv, rv2, v)):
                want, _ = RO.reorder_rotations(x[b, h].float().numpy(), L, L, R0[b, h].numpy(), 16)
                assert np.array_equal(Rg[b, h].cpu().numpy(), want), (b, h)
    res = {}
    for name, (Rk, Rv) in (("given", (rk, rv)), ("coselection", (rk2.cpu(), rv2.cpu()))):
        c = M.MosaicCache(params, ns, L, rotated=True)
        c.compress(k.cuda(), v.cuda(), [L] * ns, Rk.cuda().contiguous(), Rv.cuda().contiguous())
        st = c.stats()
        res[name] = (st["ratio"], sorted(st["strategies"]))
        for p in range(ns * hkv):
            b, h = divmod(p, hkv)
            pr = O.Pair(op, L, Rk[b, h].numpy(), Rv[b, h].numpy())
            pr.compress(bits(k[b, h]), bits(v[b, h]))
            assert_state_equal(c, p, pr, where=name)
    print(f"[coselection] ratio given {res['given']}, reordered {res['coselection']}", flush=True)
    assert {s[:2] for s in res["given"][1]} == {(16, 1)} and {s[:2] for s in res["coselection"][1]} == {(16, 4)}
    assert res["coselection"][0] > 1.25 * res["given"][0]
