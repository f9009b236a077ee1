"""CPU emulation of the fp32 HIP kernels' addressing (tests only).

Mirrors, step by step, the index arithmetic of ``conv_f32_kernel`` (family 1,
register-staged) and ``conv_f32_dma_kernel`` (family 2, direct-to-LDS loads)
for a
resolved launch geometry (``conv_fwd_geometry``): workgroup -> tile mapping
(with the XCD remap), the per-thread staging lists, LDS writes and reads of
each pipeline step, the MFMA operand lanes and the epilogue stores.  Every
global and LDS access is checked against its buffer; LDS reads by unmasked
lanes must hit data written in the same step; every output must be stored
exactly once.  The arithmetic is done in float64 so the result can be
compared with the oracle.  This lets a launch configuration be checked on the
host before it ever runs on a GPU.
"""
import numpy as np


class EmulationError(AssertionError):
    pass


def _chk(cond, msg):
    if not np.all(cond):
        raise EmulationError(msg)


DIVISORS = {"in_cstride": "in_cstride", "in_wp": "in_wp", "H": "H", "ker_rstride": "ker_rstride", "tw": "tw",
            "P": "P", "nph": "nph", "nb": "nb", "Wi": "Wi", "tiles_k": "tiles_k", "tiles_cols": "tiles_cols",
            "tiles_rows": "tiles_rows"}


def fdiv(n, g, name):
    """n // g[name] as the kernels compute it, (n * m) >> (31 + s) with the
    launch's exported multiplier; checked against floor division."""
    m, s = g[f"dv_{name}_m"], g[f"dv_{name}_s"]
    d = g[DIVISORS[name]]
    nn = np.asarray(n, dtype=np.int64)
    _chk((nn >= 0).all() and (nn < 2 ** 31).all(), f"numerator of /{name} outside [0, 2^31)")
    _chk(m > 0 and d > 0, f"launch divides by {name} without a multiplier")
    q = ((nn.astype(np.uint64) * np.uint64(m)) >> np.uint64(31 + s)).astype(np.int64)
    _chk((q == nn // d).all(), f"fast division by {name} = {d} is not exact")
    return q if np.ndim(n) else int(q)


def tile_coord(g, b, BK):
    G = g["num_tiles"]
    G8 = G & ~7
    L = (b & 7) * (G8 >> 3) + (b >> 3) if b < G8 else b
    if g["order"] == 0:
        rest = fdiv(L, g, "tiles_k")
        kt = L - rest * g["tiles_k"]
        rt = fdiv(rest, g, "tiles_cols")
        ct = rest - rt * g["tiles_cols"]
    else:
        rest = fdiv(L, g, "tiles_cols")
        ct = L - rest * g["tiles_cols"]
        kt = fdiv(rest, g, "tiles_rows")
        rt = rest - kt * g["tiles_rows"]
    NP = g["N"] * g["P"]
    rho0 = rt * g["tr"]
    rho_end = min(rho0 + g["tr"], NP)
    q0 = ct * g["tw"]
    tw_eff = min(g["tw"], g["Q"] - q0)
    k0 = kt * BK
    nf = fdiv(rho0, g, "P")
    pf = rho0 - nf * g["P"]
    nu0 = nf * g["H"] + pf
    nl = fdiv(rho_end - 1, g, "P")
    pl = rho_end - 1 - nl * g["P"]
    nrows = nl * g["H"] + pl + g["R"] - nu0
    return L, dict(rho0=rho0, rho_end=rho_end, q0=q0, tw_eff=tw_eff, k0=k0, nu0=nu0, nrows=nrows)


def emulate(g, In, Ker, wgs=None):
    """Run the kernel's addressing for workgroups ``wgs`` (default: all).

    In, Ker: flat float64 arrays of the problem (the kernel view, identical
    memory).  Returns (out_flat, written) where written counts stores per
    output element (NaN outputs where nothing was stored)."""
    if g["family"] in (4, 5):
        return emulate_stream1x1(g, In, Ker, wgs)
    if g["family"] == 7:
        return emulate_stream1x1_bal(g, In, Ker, wgs)
    N, C, K, H, W, R, S, P, Q = (g[x] for x in "N C K H W R S P Q".split())
    WK, WP, TC, KV, NT = g["wk"], g["wp"], g["tc"], g["ker_vec"], g["threads"]
    _chk(NT == 256 or (g["family"] == 2 and NT in (256, 512)), "threads per workgroup")
    nwk, nwp = g["nwk"], g["nwp"]
    NWC = g.get("nwc", 1)  # groups of waves splitting each step's channels
    _chk(nwk * nwp * NWC * 64 == NT, "waves do not fill the workgroup")
    BK = 16 * WK * nwk
    RS = R * S
    if g["rc"]:
        _chk(g["rc"] == R and g["sc"] == S, "compile-time taps differ from the shape")
    in_size, ker_size, out_size = N * C * H * W, K * C * R * S, N * K * P * Q
    # direct phase addressing (conv_fwd_ex): In is the caller's outer tensor
    nph = g.get("nph", 0)
    if nph:
        _chk(g["family"] == 2 and g["in_vec"] == 1 and g["tc"] % nph == 0, "direct phase addressing")
        _chk(nph == g["na"] * g["nb"] and C == g["C0"] * nph, "phase counts")
        in_size = N * g["C0"] * g["H0"] * g["W0"]
    # phase skip: chunks laid out phase-major in LDS (position f * TC/4 + c
    # holds phase f of the chunk's input channel c), zero-tap steps left out
    PSK = bool(g.get("phase_skip", 0))
    if PSK:
        _chk(nph == 4 and g["na"] == 2 and g["nb"] == 2 and g["sh"] == 2 and g["sw"] == 2, "four phases, stride 2")
        _chk(g["tc"] % 16 == 0 and g["in_vec"] == 1 and R * S % g["ker_vec"] == 0, "phase-skip instance")
    _chk(In.size == in_size and Ker.size == ker_size, "input sizes")
    dma = g["family"] == 2
    MF32 = bool(g.get("mfma32", 0))
    _chk(not MF32 or (dma and WK == 4 and WP % 2 == 0), "32x32x2 loop: 64-row k tile, pairs of 16-pixel units")
    NPB, BW, NKB, CG = (WP // 2, 32, 2, 2) if MF32 else (WP, 16, WK, 4)
    _chk(NWC == 1 or (dma and not MF32 and TC % (CG * NWC) == 0), "channel groups of waves")
    l32, h32 = np.arange(64) & 31, np.arange(64) >> 5
    jl = l32 if MF32 else (np.arange(64) & 15)
    chl = h32 if MF32 else (np.arange(64) >> 4)  # this lane's channel within a step's group
    NW = NT // 64
    if dma:
        NLI, NLK, KVI, NS = g["max_ni"], g["max_nk"], g["in_vec"], g["stages"]
        IN_REGION = NLI * NW * 64 * KVI
        KER_REGION = NLK * NW * 64 * KV
        _chk(g["in_region"] == IN_REGION and g["stage_elems"] == IN_REGION + KER_REGION, "DMA regions")
        _chk(NS * g["stage_elems"] * 4 == g["lds_bytes"], "LDS byte count")
        _chk(g["in_bytes"] == in_size * 4 and g["ker_bytes"] == ker_size * 4, "buffer ranges")
        _chk(in_size * 4 < 2 ** 31 and ker_size * 4 < 2 ** 31, "tensors under 2 GB")
        lin_n, lker_n = IN_REGION, KER_REGION
        _chk(TC * g["in_cstride"] <= IN_REGION, "In tile exceeds its LDS region")
        _chk(BK * g["ker_rstride"] <= KER_REGION, "Ker tile exceeds its LDS region")
    else:
        lin_n, lker_n = g["lds_in_elems"], g["lds_ker_elems"]
        _chk(2 * (lin_n + lker_n) * 4 == g["lds_bytes"], "LDS byte count")
    _chk(g["lds_bytes"] <= 160 * 1024, "LDS capacity")
    out = np.full(out_size, np.nan)
    written = np.zeros(out_size, np.int64)
    tid = np.arange(NT)
    lane = np.arange(64)
    j, gq = lane & 15, lane >> 4
    E = g["in_rows"] * g["in_wp"]
    TCRS = TC * RS
    _chk(TCRS % KV == 0, "Ker vector width")
    per_row = TCRS // KV
    if not dma:
        _chk(g["ni_in"] <= g["max_ni"] and g["ni_ker"] <= g["max_nk"], "staging capacity")
        _chk(g["ni_in"] * NT >= TC * E, "In staging does not cover the LDS tile")
        _chk(g["ni_ker"] * NT >= BK * per_row, "Ker staging does not cover the LDS tile")
    split, cps = g["split"], g["cps"]
    _chk(split >= 1 and (split == 1 or dma), "only the direct-to-LDS kernel splits the reduction")
    _chk(g["grid"] == g["num_tiles"] * split, "workgroups = tiles x channel ranges")
    _chk(split * cps >= g["nchunks"] and (split - 1) * cps < g["nchunks"], "channel ranges cover the steps")
    # a split plan writes range r's partial sums to workspace slice r; the
    # second pass adds the slices in range order
    ws = np.full(split * out_size, np.nan) if split > 1 else None
    ws_written = np.zeros(split * out_size, np.int64) if split > 1 else None
    seen_L = set()
    tiles = range(g["num_tiles"]) if wgs is None else wgs
    for b in [r * g["num_tiles"] + tb for tb in tiles for r in range(split)]:
        split_r, tb = divmod(b, g["num_tiles"])
        L, t = tile_coord(g, tb, BK)
        _chk(0 <= L < g["num_tiles"] and (L, split_r) not in seen_L, "workgroup remap is not a bijection")
        seen_L.add((L, split_r))
        ncols = t["tw_eff"] + S - 1
        _chk(t["nrows"] <= g["in_rows"], "tile needs more LDS rows than allocated")
        # In staging list
        in_items = []
        for i in range(g["max_ni"]):
            idx = tid + NT * i
            ok = (i < g["ni_in"]) & (idx < TC * E)
            cl, e = idx // E, idx % E
            row, x = e // g["in_wp"], e % g["in_wp"]
            loff = cl * g["in_cstride"] + e
            inside = ok & (row < t["nrows"]) & (x < ncols)
            nu = t["nu0"] + row
            n, y = nu // H, nu % H
            goff = np.where(inside, ((n * C + cl) * H + y) * W + t["q0"] + x, -1)
            _chk(~ok | (loff < (1 << 20)), "LDS offset does not fit its packing")
            in_items.append((ok, cl, loff, goff))
        ker_items = []
        for i in range(g["max_nk"]):
            idx = tid + NT * i
            ok = (i < g["ni_ker"]) & (idx < BK * per_row)
            kl, m = idx // per_row, (idx % per_row) * KV
            ker_items.append((ok, kl, m))
        # per-lane pixel offsets and Ker rows, per wave (32x32x2 loop: 32-pixel
        # blocks and 32-row k blocks, lane (l32, h32))
        tpx = g["tr"] * g["tw"]
        waves = []
        for wave in range(nwk * nwp * NWC):
            wg, wc = wave % (nwk * nwp), wave // (nwk * nwp)
            wk, wp = wg % nwk, wg // nwk
            poff, pvalid, pinfo = [], [], []
            for pb in range(NPB):
                px = wp * WP * 16 + pb * BW + jl
                if dma:
                    row_i = fdiv(px, g, "tw")
                    col = px - row_i * g["tw"]
                else:
                    row_i, col = px // g["tw"], px % g["tw"]
                rho = t["rho0"] + row_i
                valid = (px < tpx) & (rho < t["rho_end"]) & (col < t["tw_eff"])
                if dma:
                    n = fdiv(rho, g, "P")
                    p = rho - n * P
                else:
                    n, p = rho // P, rho % P
                off = np.where(valid, (n * H + p - t["nu0"]) * g["in_wp"] + col, 0)
                poff.append(off)
                pvalid.append(valid)
                pinfo.append((n, p, col))
            if MF32:
                koff = [(wk * 64 + kb * 32 + l32) * g["ker_rstride"] for kb in range(NKB)]
            else:
                koff = [((wk * WK + kb) * 16 + j) * g["ker_rstride"] for kb in range(NKB)]
            waves.append(dict(wk=wk, wp=wp, wg=wg, wc=wc, poff=poff, pvalid=pvalid, pinfo=pinfo, koff=koff,
                              acc=np.zeros((NKB, NPB, BW, BW))))
        lin = [np.full(lin_n, np.nan), np.full(lin_n, np.nan)]
        lker = [np.full(lker_n, np.nan), np.full(lker_n, np.nan)]

        def stage_dma(c0, buf):
            wave = tid >> 6
            lane_t = tid & 63
            fresh_in = np.full(lin_n, np.nan)
            for i in range(NLI):
                e = ((i * NW + wave) * 64 + lane_t) * KVI
                cl = fdiv(e, g, "in_cstride")
                pos = e - cl * g["in_cstride"]
                row = fdiv(pos, g, "in_wp")
                x = pos - row * g["in_wp"]
                valid = (e < TC * g["in_cstride"]) & (row < t["nrows"]) & (x < ncols) & (c0 + cl < C)
                nu = t["nu0"] + row
                n = fdiv(nu, g, "H")
                y = nu - n * H
                if nph:
                    # chunk-local input channel and phase, as the kernel splits them
                    _chk(c0 % nph == 0, "a pipeline step splits a channel's phases")
                    if PSK:
                        cr, f = cl % (TC // 4), cl // (TC // 4)
                        # the channel-count check on the inner channel
                        valid = (e < TC * g["in_cstride"]) & (row < t["nrows"]) & (x < ncols) & (c0 + cr * 4 + f < C)
                    else:
                        cr = fdiv(cl, g, "nph")
                        f = cl - cr * nph
                    a = fdiv(f, g, "nb")
                    b = f - a * g["nb"]
                    yi, xi = y, t["q0"] + x
                    if g["Wi"]:  # 1x1 kernel view: one row of H' x W' pixels per image
                        yi = fdiv(xi, g, "Wi")
                        xi = xi - yi * g["Wi"]
                    iy, ix = yi * g["sh"] + a - g["ph"], xi * g["sw"] + b - g["pw"]
                    valid = valid & (iy >= 0) & (iy < g["H0"]) & (ix >= 0) & (ix < g["W0"])
                    goff = ((n * g["C0"] + cr) * g["H0"] + iy) * g["W0"] + ix
                    coff = fdiv(c0, g, "nph") * g["H0"] * g["W0"]
                else:
                    goff = ((n * C + cl) * H + y) * W + t["q0"] + x
                    coff = c0 * H * W
                for q in range(KVI):
                    src = coff + goff + q
                    _chk((src[valid] >= 0) & (src[valid] < in_size), "In read out of bounds")
                    _chk(~valid | (src * 4 < 2 ** 31), "In byte offset overflows")
                    vals = np.where(valid, In[np.clip(src, 0, in_size - 1)], 0.0)
                    dst = e + q
                    _chk(dst < lin_n, "In DMA writes past its region")
                    _chk(np.isnan(fresh_in[dst]), "two lanes write one LDS In element")
                    fresh_in[dst] = vals
            lin[buf][:] = fresh_in
            fresh_k = np.full(lker_n, np.nan)
            mlim = (C - c0) * RS
            for i in range(NLK):
                e = ((i * NW + wave) * 64 + lane_t) * KV
                kl = fdiv(e, g, "ker_rstride")
                m = e - kl * g["ker_rstride"]
                if PSK:  # LDS position (f * TC/4 + c) * RS + rs <- inner channel c * 4 + f
                    m = ((m // RS) % (TC // 4) * 4 + (m // RS) // (TC // 4)) * RS + m % RS
                    valid = (kl < BK) & (e - kl * g["ker_rstride"] < TCRS) & (t["k0"] + kl < K) & (m < mlim)
                else:
                    valid = (kl < BK) & (m < TCRS) & (t["k0"] + kl < K) & (m < mlim)
                if KV > 1:
                    _chk(~valid | (m + KV <= mlim), "Ker vector straddles the channel range")
                    _chk(g["ker_rstride"] % KV == 0, "Ker vector straddles an LDS row")
                for q in range(KV):
                    src = (t["k0"] + kl) * C * RS + c0 * RS + m + q
                    _chk((src[valid] >= 0) & (src[valid] < ker_size), "Ker read out of bounds")
                    vals = np.where(valid, Ker[np.clip(src, 0, ker_size - 1)], 0.0)
                    dst = e + q
                    _chk(dst < lker_n, "Ker DMA writes past its region")
                    _chk(~valid | (m % RS + q < RS) if PSK else True, "phase-skip Ker vector leaves its channel")
                    _chk(np.isnan(fresh_k[dst]), "two lanes write one LDS Ker element")
                    fresh_k[dst] = vals
            lker[buf][:] = fresh_k

        def stage(c0, buf):
            if dma:
                return stage_dma(c0, buf)
            fresh_in = np.full(lin_n, np.nan)
            for ok, cl, loff, goff in in_items:
                use = ok
                src = np.where(use & (goff >= 0) & (c0 + cl < C), c0 * H * W + goff, -1)
                _chk(src[src >= 0] < in_size, "In read out of bounds")
                vals = np.where(src >= 0, In[np.clip(src, 0, in_size - 1)], 0.0)
                _chk(loff[use] < lin_n, "LDS In write out of bounds")
                _chk(np.isnan(fresh_in[loff[use]]), "two threads write one LDS In element")
                fresh_in[loff[use]] = vals[use]
            lin[buf][:] = fresh_in  # anything not rewritten this step counts as stale
            fresh_k = np.full(lker_n, np.nan)
            mlim = (C - c0) * RS
            for ok, kl, m in ker_items:
                valid = ok & (t["k0"] + kl < K) & (m < mlim)
                base = c0 * RS + (t["k0"] + kl) * C * RS + m
                for e in range(KV):
                    src = np.where(valid, base + e, -1)
                    _chk(src[valid] < ker_size, "Ker read out of bounds")
                    vals = np.where(valid, Ker[np.clip(src, 0, ker_size - 1)], 0.0)
                    dst = kl * g["ker_rstride"] + m + e
                    _chk(dst[ok] < lker_n, "LDS Ker write out of bounds")
                    _chk(np.isnan(fresh_k[dst[ok]]), "two threads write one LDS Ker element")
                    fresh_k[dst[ok]] = vals[ok]
            lker[buf][:] = fresh_k

        def compute(buf):
            for wv in waves:
                per = TC // CG // NWC  # channel groups of this wave's slice
                for cs in range(wv["wc"] * per, (wv["wc"] + 1) * per):
                    for r in range(R):
                        for s in range(S):
                            if PSK:
                                f = cs * CG // (TC // 4)  # the group's phase (a, b)
                                if (f >> 1 == 1 and r == R - 1) or (f & 1 == 1 and s == S - 1):
                                    continue  # a zero tap of this phase: the kernel leaves the step out
                            tap = r * g["in_wp"] + s
                            rs = r * S + s
                            A = []
                            for kb in range(NKB):
                                ai = (cs * CG + chl) * RS + wv["koff"][kb] + rs
                                _chk((ai >= 0) & (ai < lker_n), "LDS Ker read out of bounds")
                                a = lker[buf][ai]
                                _chk(~np.isnan(a), "LDS Ker read of an element not staged this step")
                                A.append(a)
                            for pb in range(NPB):
                                bi = (cs * CG + chl) * g["in_cstride"] + wv["poff"][pb] + tap
                                _chk((bi >= 0) & (bi < lin_n), "LDS In read out of bounds")
                                bv = lin[buf][bi]
                                _chk(~np.isnan(bv), "LDS In read of an element not staged this step")
                                Bm = np.zeros((CG, BW))
                                Bm[chl, jl] = bv
                                for kb in range(NKB):
                                    Am = np.zeros((BW, CG))
                                    Am[jl, chl] = A[kb]
                                    wv["acc"][kb, pb] += Am @ Bm

        ch0 = split_r * cps
        nch = min(cps, g["nchunks"] - ch0)
        _chk(nch >= 1, "empty channel range")
        stage(ch0 * TC, 0)
        for ch in range(nch):
            compute(ch & 1)
            if ch + 1 < nch:
                stage((ch0 + ch + 1) * TC, (ch + 1) & 1)
        if NWC > 1:
            # accumulators parked in LDS per wave and register, summed over
            # the groups in order; wave (wg, wc) stores registers
            # [wc * NREG / NWC, (wc + 1) * NREG / NWC)
            NREG = NKB * NPB * 4
            _chk(NREG % NWC == 0, "registers per group")
            _chk(NT // 64 * NREG * 64 <= g["stages"] * g["stage_elems"], "reduction exceeds the LDS")
            NG = nwk * nwp
            for wg in range(NG):
                tot = waves[wg]["acc"].copy()
                for c in range(1, NWC):
                    tot = tot + waves[c * NG + wg]["acc"]
                for c in range(NWC):
                    waves[c * NG + wg]["red"] = tot
                    waves[c * NG + wg]["regs"] = set(range(c * NREG // NWC, (c + 1) * NREG // NWC))
        for wv in waves:
            for pb in range(NPB):
                valid = wv["pvalid"][pb]
                n, p, col = wv["pinfo"][pb]
                for kb in range(NKB):
                    for v in range(16 if MF32 else 4):
                        if NWC > 1 and (kb * NPB + pb) * 4 + v not in wv["regs"]:
                            continue
                        if MF32:
                            i = 8 * (v // 4) + 4 * h32 + v % 4
                            k = t["k0"] + wv["wk"] * 64 + kb * 32 + i
                        else:
                            i = 4 * gq + v
                            k = t["k0"] + (wv["wk"] * WK + kb) * 16 + i
                        st = valid & (k < K)
                        dst = ((n * K + k) * P + p) * Q + t["q0"] + col
                        _chk((dst[st] >= 0) & (dst[st] < out_size), "Out store out of bounds")
                        vals = (wv["red"] if NWC > 1 else wv["acc"])[kb, pb][i, jl]
                        if split > 1:
                            wdst = split_r * out_size + dst
                            ws[wdst[st]] = vals[st]
                            np.add.at(ws_written, wdst[st], 1)
                        else:
                            out[dst[st]] = vals[st]
                            np.add.at(written, dst[st], 1)
    if split > 1:
        per = ws_written.reshape(split, out_size)
        touched = per.max(axis=0) > 0
        # every slice of every touched output written exactly once
        _chk((per[:, touched] == 1).all(), "a channel range stored an output twice or not at all")
        sl = ws.reshape(split, out_size)
        acc = sl[0].copy()
        for r in range(1, split):
            acc = acc + sl[r]
        out = np.where(touched, acc, np.nan)
        written = touched.astype(np.int64)
    return out, written


# ---------------------------------------------------------------------------
# bf16 family (conv_bf16_kernel): persistent workgroups over every G-th tile,
# channel-fastest swizzled LDS images, 16x16x32 MFMA.

def _swz(chunk, idx):
    return chunk ^ ((idx >> 1) & 3)


def emulate_bf16(g, In, Ker, wgs=None, in_aligned=True, out_aligned=True, out_bf16=False):
    """In, Ker: flat float64 arrays holding the bf16 values.  Emulates the
    workgroups ``wgs`` (default all) of the persistent grid."""
    if g["family"] == 6:
        return emulate_bf16_tr(g, In, Ker, wgs, out_aligned, out_bf16)
    N, C, K, H, W, R, S, P, Q = (g[x] for x in "N C K H W R S P Q".split())
    _chk(g["family"] == 3 and g["threads"] == 256, "bf16 family geometry")
    WK, WP, MAXIT = g["wk"], g["wp"], g["max_ni"]
    nwk, nwp = g["nwk"], g["nwp"]
    _chk(nwk * nwp == 4, "waves")
    BK = 16 * WK * nwk
    RS = R * S
    TC = 32
    kpitch = RS if RS % 2 else RS + 1
    _chk(g["ker_rstride"] == kpitch, "Ker pitch")
    in_wp = g["in_wp"]
    _chk(in_wp % 2 == 0, "halo pitch even")
    lds_bytes = BK * kpitch * 64 + g["in_rows"] * in_wp * 64
    _chk(lds_bytes == g["stage_elems"] == g["lds_bytes"] and lds_bytes <= 160 * 1024, "LDS bytes")
    in_size, ker_size, out_size = N * C * H * W, K * C * RS, N * K * P * Q
    _chk(In.size == in_size and Ker.size == ker_size, "input sizes")
    out = np.full(out_size, np.nan)
    written = np.zeros(out_size, np.int64)
    tiles = g["tiles_rows"] * g["tiles_cols"] * g["tiles_k"]
    G = g["grid"]
    _chk(1 <= G <= tiles, "grid")
    nchunks = -(-C // TC)
    resident = nchunks == 1 and g["tiles_k"] == 1
    npair = in_wp // 2
    in_items = 4 * g["in_rows"] * npair
    _chk(in_items <= MAXIT * 256, "In staging capacity")
    tid = np.arange(256)
    lane = np.arange(64)
    j, gq = lane & 15, lane >> 4
    seen = np.zeros(tiles, bool)
    for b in (range(G) if wgs is None else wgs):
        G8 = G & ~7
        L = (b & 7) * (G8 >> 3) + (b >> 3) if b < G8 else b
        lds = np.full(lds_bytes // 2, np.nan)  # bf16 slots

        def stage_ker(k0, c0):
            items = BK * RS * 4
            for it in range(items):
                o, rest = it & 3, it >> 2
                rs, kl = rest % RS, rest // RS
                for e in range(8):
                    c, k = c0 + 8 * o + e, k0 + kl
                    val = 0.0
                    if c < C and k < K:
                        src = (k * C + c) * RS + rs
                        _chk(0 <= src < ker_size, "Ker read out of bounds")
                        val = Ker[src]
                    dst = ((kl * kpitch + rs) * 64 + _swz(o, kl) * 16) // 2 + e
                    _chk(dst < BK * kpitch * 32, "LDS Ker write out of range")
                    lds[dst] = val

        def stage_in(T, c0):
            kt, rest = T % g["tiles_k"], T // g["tiles_k"]
            ct, rt = rest % g["tiles_cols"], rest // g["tiles_cols"]
            NP = N * P
            rho0, rho_end = rt * g["tr"], min(rt * g["tr"] + g["tr"], NP)
            q0 = ct * g["tw"]
            ncols = min(g["tw"], Q - q0) + S - 1
            nf = rho0 // P
            nu0 = nf * H + (rho0 - nf * P)
            nl = (rho_end - 1) // P
            nrows = nl * H + (rho_end - 1 - nl * P) + R - nu0
            _chk(nrows <= g["in_rows"], "tile needs more halo rows than allocated")
            ker_base = BK * kpitch * 32
            for m in range(MAXIT):
                it = tid + m * 256
                o = it // (g["in_rows"] * npair)
                rest = it - o * (g["in_rows"] * npair)
                row, x = rest // npair, (rest - (rest // npair) * npair) * 2
                for t in range(256):
                    if it[t] >= in_items:
                        continue
                    ok = row[t] < nrows
                    nu = nu0 + row[t]
                    n, y = nu // H, nu % H
                    for e in range(8):
                        c = c0 + 8 * o[t] + e
                        for d in range(2):
                            xx = x[t] + d
                            val = 0.0
                            if ok and c < C and xx < ncols:
                                src = ((n * C + c) * H + y) * W + q0 + xx
                                _chk(0 <= src < in_size, "In read out of bounds")
                                val = In[src]
                            px = row[t] * in_wp + x[t] + d
                            dst = ker_base + (px * 64 + _swz(o[t], px) * 16) // 2 + e
                            _chk(dst < lds.size, "LDS In write out of range")
                            lds[dst] = val
            return rho0, rho_end, q0, kt, nu0

        if resident:
            stage_ker(0, 0)
        for T in range(L, tiles, G):  # tiles L, L + G, ...
            _chk(not seen[T], "tile processed twice")
            seen[T] = True
            acc = {}
            for ch in range(nchunks):
                if not resident:
                    kt0 = T % g["tiles_k"]
                    stage_ker(kt0 * BK, ch * TC)
                rho0, rho_end, q0, kt, nu0 = stage_in(T, ch * TC)
                k0 = kt * BK
                tw_eff = min(g["tw"], Q - q0)
                tpx = g["tr"] * g["tw"]
                for wave in range(4):
                    wk, wp = wave % nwk, wave // nwk
                    for pb in range(WP):
                        px = (wp * WP + pb) * 16 + j
                        row_i, col = px // g["tw"], px % g["tw"]
                        rho = rho0 + row_i
                        valid = (px < tpx) & (rho < rho_end) & (col < tw_eff)
                        n, p = rho // P, rho % P
                        poff = np.where(valid, (n * H + p - nu0) * in_wp + col, 0)
                        for kb in range(WK):
                            kl = (wk * WK + kb) * 16 + j
                            cmat = acc.setdefault((wave, kb, pb), np.zeros((16, 16)))
                            for r in range(R):
                                for s in range(S):
                                    ai = ((kl * kpitch + r * S + s) * 64 + _swz(gq, kl) * 16) // 2
                                    pp = poff + r * in_wp + s
                                    bi = BK * kpitch * 32 + (pp * 64 + _swz(gq, pp) * 16) // 2
                                    A = np.zeros((16, 32))
                                    Bm = np.zeros((32, 16))
                                    for e in range(8):
                                        _chk((ai + e < BK * kpitch * 32).all(), "LDS Ker read range")
                                        _chk((bi + e < lds.size).all(), "LDS In read range")
                                        av = lds[ai + e]
                                        bv = lds[bi + e]
                                        _chk(~np.isnan(av), "Ker read of an unstaged slot")
                                        _chk(~np.isnan(bv[valid]), "In read of an unstaged slot")
                                        A[j, 8 * gq + e] = av
                                        Bm[8 * gq + e, j] = np.nan_to_num(bv)
                                    cmat += A @ Bm
            # epilogue
            for wave in range(4):
                wk, wp = wave % nwk, wave // nwk
                for pb in range(WP):
                    px = (wp * WP + pb) * 16 + j
                    row_i, col = px // g["tw"], px % g["tw"]
                    rho = rho0 + row_i
                    valid = (px < tpx) & (rho < rho_end) & (col < tw_eff)
                    n, p = rho // P, rho % P
                    for kb in range(WK):
                        for v in range(4):
                            k = k0 + (wk * WK + kb) * 16 + 4 * gq + v
                            st = valid & (k < K)
                            dst = ((n * K + k) * P + p) * Q + q0 + col
                            _chk((dst[st] >= 0).all() and (dst[st] < out_size).all(), "Out store range")
                            out[dst[st]] = acc[(wave, kb, pb)][4 * gq + v, j][st]
                            np.add.at(written, dst[st], 1)
    return out, written


# ---------------------------------------------------------------------------
# Pointwise streaming family (conv1x1_stream_kernel).

def emulate_stream1x1(g, In, Ker, wgs=None):
    """The pointwise streaming kernels.

    Family 4 (unrolled for C = tc): per SIMD a wave of max_ni and (if
    max_nk > 0) a second wave of max_nk units of 16 pixels; a wave with U
    units does U//2 blocks of 32 pixels on 32x32x2 MFMAs (two 32-row k
    blocks, channel pairs) and U%2 blocks of 16 on 16x16x4 MFMAs; Ker rows
    copied to LDS in 64-channel chunks.  Family 5 (looped over trips of `stages` quads): max_ni then
    max_nk blocks of 16 pixels, Ker zero-padded to whole trips.  Ker rows
    [k][c] in LDS with a pitch of the stored channel count + 1; In operands
    from raw buffer loads whose 32-bit byte offsets are emulated exactly
    (offsets at or past the buffer size read 0)."""
    N, C, K, H, W = (g[x] for x in "N C K H W".split())
    fam = g["family"]
    _chk(fam in (4, 5) and g["R"] == 1 and g["S"] == 1, "stream geometry")
    HW = W  # kernel view: one row per image
    _chk(H == 1, "kernel view of a pointwise layer")
    _chk(C % 4 == 0, "whole channel quads")
    D = g["stages"]
    nq = C // 4
    if fam == 4:
        _chk(g["tc"] == C and nq % 16 == 0, "unrolled instance for this channel count")
        UA, UB = g["max_ni"], g["max_nk"]
        NW = 8 if UB > 0 else 4
        _chk(g["threads"] == 64 * NW, "threads per workgroup")
        NB = UA + UB
        nq_run, cst = nq, C
    else:
        _chk(g["tc"] == 0 and g["threads"] == 256, "looped instance")
        NB1, NB2 = g["max_ni"], g["max_nk"]
        NB = NB1 + NB2
        nq_run = -(-nq // D) * D
        cst = 4 * nq_run
    _chk(g["wp"] == NB, "pixel blocks per wave")
    pitch = cst + 1
    wpx = g["tw"]
    _chk(1 <= wpx <= 16 * NB, "pixels per wave")
    _chk(g["stage_elems"] == 64 * pitch * 4 == g["lds_bytes"] and g["lds_bytes"] <= 160 * 1024, "LDS bytes")
    total_px = N * HW
    in_size, ker_size, out_size = N * C * HW, K * C, N * K * HW
    _chk(In.size == in_size and Ker.size == ker_size, "input sizes")
    _chk(g["in_bytes"] == in_size * 4 and in_size * 4 < 2 ** 30, "In byte range below 1 GB")
    _chk(g["ker_bytes"] == ker_size * 4 and ker_size * 4 < 2 ** 31, "Ker byte range below the sentinel")
    out = np.full(out_size, np.nan)
    written = np.zeros(out_size, np.int64)
    lane = np.arange(64)
    KOOB, QOOB, M32 = 0x80000000, 0x40000000, 0xFFFFFFFF

    def in_load(voff, byte_add, expect):
        off = (voff + byte_add) & M32
        hit = off < g["in_bytes"]
        _chk((off[hit] % 4 == 0).all(), "misaligned In offset")
        # the range check must drop exactly the masked lanes (and padded quads)
        _chk((hit == expect).all(), "range check does not match the mask")
        return np.where(hit, In[np.where(hit, off // 4, 0)], 0.0)

    def lds_read(lds, idx):
        _chk((idx >= 0).all() and (idx < lds.size).all(), "LDS Ker read out of range")
        v = lds[idx]
        _chk(not np.isnan(v).any(), "LDS Ker read of an unwritten element")
        return v

    def store(acc_rows, k, px, valid):
        n, hw = px // HW, px % HW
        st = valid & (k < K)
        dst = (n * K + k) * HW + hw
        _chk((dst[st] >= 0).all() and (dst[st] < out_size).all(), "Out store range")
        out[dst[st]] = acc_rows[st]
        np.add.at(written, dst[st], 1)

    def block16(lds, k0, px_begin, px_end, blk_px0, quads):
        """One 16-pixel block on 16x16x4 MFMAs (lane (j, gq))."""
        j, gq = lane & 15, lane >> 4
        px = blk_px0 + j
        valid = px < px_end
        n, hw = px // HW, px % HW
        voff = np.where(valid, ((n * C + gq) * HW + hw) * 4, KOOB)
        acc = np.zeros((4, 16, 16))
        for q in range(quads):
            bv = in_load(voff, q * 16 * HW + (0 if q < nq else QOOB), valid & (q < nq))
            for kb in range(4):
                av = lds_read(lds, (kb * 16 + j) * pitch + 4 * q + gq)
                Am = np.zeros((16, 4))
                Am[j, gq] = av
                Bm = np.zeros((4, 16))
                Bm[gq, j] = bv
                acc[kb] += Am @ Bm
        for kb in range(4):
            for v in range(4):
                store(acc[kb][4 * gq + v, j], k0 + kb * 16 + 4 * gq + v, px, valid)

    def block32(lds, k0, px_end, blk_px0):
        """One 32-pixel block on 32x32x2 MFMAs (lane (l32, h32))."""
        l32, h32 = lane & 31, lane >> 5
        px = blk_px0 + l32
        valid = px < px_end
        n, hw = px // HW, px % HW
        voff = np.where(valid, ((n * C + h32) * HW + hw) * 4, KOOB)
        acc = np.zeros((2, 32, 32))
        for q in range(nq):
            for e in range(2):
                bv = in_load(voff, (4 * q + 2 * e) * 4 * HW, valid)
                for kb in range(2):
                    av = lds_read(lds, (kb * 32 + l32) * pitch + 4 * q + 2 * e + h32)
                    Am = np.zeros((32, 2))
                    Am[l32, h32] = av
                    Bm = np.zeros((2, 32))
                    Bm[h32, l32] = bv
                    acc[kb] += Am @ Bm
        for kb in range(2):
            for v in range(16):
                i = 8 * (v // 4) + 4 * h32 + v % 4
                store(acc[kb][i, l32], k0 + 32 * kb + i, px, valid)

    for b in (range(g["grid"]) if wgs is None else wgs):
        kt, pg = b % g["tiles_k"], b // g["tiles_k"]
        k0 = kt * 64
        lds = np.full(64 * pitch, np.nan)  # the pad column is never read
        if fam == 4:
            # wave w copies rows (64/NW)w .. (64/NW)(w+1)-1, 64 channels per
            # load: LDS destination M0 + 4 * lane, source offset or the sentinel
            for w in range(NW):
                for ch in range(C // 64):
                    for i in range(64 // NW):
                        kl = w * (64 // NW) + i
                        k = k0 + kl
                        dst = kl * pitch + ch * 64 + lane
                        _chk(dst.max() < lds.size, "LDS Ker chunk out of range")
                        off = (k * C + ch * 64 + lane) * 4 if k < K else np.full(64, KOOB)
                        hit = off < g["ker_bytes"]
                        _chk(hit.all() == (k < K), "Ker range check does not match the row mask")
                        lds[dst] = np.where(hit, Ker[np.where(hit, off // 4, 0)], 0.0)
        else:
            for e in range(64 * cst):
                kl, c = divmod(e, cst)
                k = k0 + kl
                lds[kl * pitch + c] = Ker[k * C + c] if (k < K and c < C) else 0.0
        for simd in range(4):
            px_begin = (pg * 4 + simd) * wpx
            px_end = min(px_begin + wpx, total_px)
            if fam == 4:
                # first wave: UA units from the SIMD's start; second: UB units after them
                for u, w_begin, w_end in ((UA, px_begin, min(px_begin + 16 * UA, px_end)),
                                          (UB, px_begin + 16 * UA, px_end)):
                    for bb in range(u // 2):
                        block32(lds, k0, w_end, w_begin + 32 * bb)
                    if u % 2:
                        block16(lds, k0, w_begin, w_end, w_begin + 32 * (u // 2), nq)
            else:
                for bb in range(NB):
                    block16(lds, k0, px_begin, px_end, px_begin + 16 * bb, nq_run)
    return out, written


def emulate_stream1x1_bal(g, In, Ker, wgs=None):
    """The balanced pointwise kernel (family 7, conv1x1_bal_kernel).

    PW = tw with 128 NB < PW <= 128 NB + 16 (NB = max_ni) sets the grid,
    G = ceil(pixels / PW) workgroups per k tile; workgroup p takes 128-pixel
    block j at (j G + p) 128 and the 16-pixel tail at NB G 128 + 16 p, pixels
    past the end masked.  Ker rows [k][c] go to LDS
    (pitch C + 1) from 16-byte loads: lane (wave, i, lane) row
    16 wave + 4 i + lane // 16, channels 64 ch + 4 (lane % 16) .. + 3.
    Wave s computes the 32-pixel blocks at (j G + p) 128 + 32 s, j < NB, on
    32x32x2 MFMAs, even and odd channel pairs in separate accumulators added
    at the store, and k rows 16 s .. 16 s + 15 of the tail block on 16x16x4
    MFMAs.  In offsets are 32-bit byte offsets from
    raw buffer loads (offsets at or past the buffer size read 0); every block
    but the last is stored during the next block, results 32 q / nq ..
    32 (q + 1) / nq - 1 at its step q, through 32-bit byte offsets of raw
    buffer stores (past Out's size: dropped), the last through pointers.
    With g["nph"] (conv_fwd_ex, one phase) In is the caller's outer tensor,
    read through the phase mapping: inner pixel (yi, xi) is In pixel
    (yi sh - ph, xi sw - pw), zero outside the image."""
    N, C, K, H, W = (g[x] for x in "N C K H W".split())
    _chk(g["family"] == 7 and g["R"] == 1 and g["S"] == 1 and H == 1, "balanced pointwise geometry")
    nph = g.get("nph", 0)
    if nph:
        _chk(nph == 1 and g["na"] == 1 and g["nb"] == 1 and g["C0"] == C and g["Wi"] > 0 and W % g["Wi"] == 0,
             "one phase of a 1x1 layer")
    _chk(g["threads"] == 256 and g["nwp"] == 4 and g["nwk"] == 1, "four waves per workgroup")
    NB = g["max_ni"]
    _chk(g["tc"] == C and C % 64 == 0 and g["wp"] == 2 * NB + 1, "instance for this channel count")
    HW = W
    nq = C // 4
    pitch = C + 1
    pw = g["tw"]
    _chk(128 * NB < pw <= 128 * NB + 16, "pixels per workgroup")
    _chk(g["stage_elems"] == 64 * pitch * 4 == g["lds_bytes"] and g["lds_bytes"] <= 160 * 1024, "LDS bytes")
    total_px = N * HW
    _chk(g["tiles_rows"] == -(-total_px // pw) and g["grid"] == g["tiles_rows"] * g["tiles_k"], "grid")
    in_size, ker_size, out_size = N * C * HW, K * C, N * K * HW
    if nph:
        in_size = N * C * g["H0"] * g["W0"]
    _chk(In.size == in_size and Ker.size == ker_size, "input sizes")
    _chk(g["in_bytes"] == in_size * 4 and in_size * 4 < 2 ** 30, "In byte range below 1 GB")
    _chk(g["ker_bytes"] == ker_size * 4 and ker_size * 4 < 2 ** 31, "Ker byte range below the sentinel")
    out = np.full(out_size, np.nan)
    written = np.zeros(out_size, np.int64)
    lane = np.arange(64)
    KOOB, M32 = 0x80000000, 0xFFFFFFFF
    out_bytes = out_size * 4
    _chk(out_bytes < 2 ** 31, "Out byte range below 2 GB")
    cstride = 4 * (g["H0"] * g["W0"] if nph else HW)

    def in_load(voff, byte_add, expect):
        off = (voff + byte_add) & M32
        hit = off < g["in_bytes"]
        _chk((off[hit] % 4 == 0).all(), "misaligned In offset")
        _chk((hit == expect).all(), "range check does not match the mask")
        return np.where(hit, In[np.where(hit, off // 4, 0)], 0.0)

    def lds_read(lds, idx):
        _chk((idx >= 0).all() and (idx < lds.size).all(), "LDS Ker read out of range")
        v = lds[idx]
        _chk(not np.isnan(v).any(), "LDS Ker read of an unwritten element")
        return v

    def store(vals, k, px, valid):
        n, hw = px // HW, px % HW
        st = valid & (k < K)
        dst = (n * K + k) * HW + hw
        _chk((dst[st] >= 0).all() and (dst[st] < out_size).all(), "Out store range")
        out[dst[st]] = vals[st]
        np.add.at(written, dst[st], 1)

    def store_buffer(vals, k, px, valid):
        # pend_base + k * HW * 4, or the sentinel for masked lanes and rows
        n, hw = px // HW, px % HW
        base = np.where(valid, (n * K * HW + hw) * 4, KOOB)
        off = np.where(k < K, base + k * HW * 4, KOOB) & M32
        hit = off < out_bytes
        _chk((hit == (valid & (k < K))).all(), "Out range check does not match the mask")
        _chk((off[hit] % 4 == 0).all(), "misaligned Out offset")
        out[off[hit] // 4] = vals[hit]
        np.add.at(written, off[hit] // 4, 1)

    def in_off(px, c, pend):
        n, hw = px // HW, px % HW
        if not nph:
            return np.where(px < pend, ((n * C + c) * HW + hw) * 4, KOOB), px < pend
        yi, xi = hw // g["Wi"], hw % g["Wi"]
        iy, ix = yi * g["sh"] - g["ph"], xi * g["sw"] - g["pw"]
        inside = (px < pend) & (iy >= 0) & (iy < g["H0"]) & (ix >= 0) & (ix < g["W0"])
        off = ((n * g["C0"] + c) * g["H0"] + iy) * g["W0"] + ix
        return np.where(inside, off * 4, KOOB), inside

    for b in (range(g["grid"]) if wgs is None else wgs):
        kt, pg = b % g["tiles_k"], b // g["tiles_k"]
        k0 = kt * 64
        GP = g["tiles_rows"]
        pend = total_px
        lds = np.full(64 * pitch, np.nan)  # the pad column is never read
        for wave in range(4):
            for ch in range(C // 64):
                for i in range(4):
                    row = 16 * wave + 4 * i + (lane >> 4)
                    k = k0 + row
                    off = np.where(k < K, (k * C + ch * 64 + 4 * (lane & 15)) * 4, KOOB)
                    hit = off < g["ker_bytes"]
                    _chk((hit == (k < K)).all(), "Ker range check does not match the row mask")
                    _chk((off[hit] % 16 == 0).all(), "Ker 16-byte load misaligned")
                    for e in range(4):
                        dst = row * pitch + ch * 64 + 4 * (lane & 15) + e
                        _chk(dst.max() < lds.size, "LDS Ker write out of range")
                        lds[dst] = np.where(hit, Ker[np.where(hit, off // 4 + e, 0)], 0.0)
        l32, h32 = lane & 31, lane >> 5
        l16, h16 = lane & 15, lane >> 4
        for wave in range(4):
            pending = None  # the previous block's 32 results, lane pixels and mask
            for j in range(NB):
                px = (j * GP + pg) * 128 + 32 * wave + l32
                voff, inside = in_off(px, h32, pend)
                valid = px < pend
                acc = np.zeros((2, 2, 32, 32))  # [kb][e]
                for q in range(nq):
                    if pending is not None:
                        vals, ppx, pvalid = pending
                        for r in range(32 * q // nq, 32 * (q + 1) // nq):
                            kb, v = r // 16, r % 16
                            store_buffer(vals[r], k0 + 32 * kb + 8 * (v // 4) + 4 * h32 + v % 4, ppx, pvalid)
                    for e in range(2):
                        bv = in_load(voff, (4 * q + 2 * e) * cstride, inside)
                        for kb in range(2):
                            av = lds_read(lds, (kb * 32 + l32) * pitch + 4 * q + 2 * e + h32)
                            Am = np.zeros((32, 2))
                            Am[l32, h32] = av
                            Bm = np.zeros((2, 32))
                            Bm[h32, l32] = bv
                            acc[kb, e] += Am @ Bm
                res = [acc[kb, 0][8 * (v // 4) + 4 * h32 + v % 4, l32] + acc[kb, 1][8 * (v // 4) + 4 * h32 + v % 4, l32]
                       for kb in range(2) for v in range(16)]
                if j < NB - 1:
                    pending = (res, px, valid)
                else:
                    for kb in range(2):
                        for v in range(16):
                            store(res[16 * kb + v], k0 + 32 * kb + 8 * (v // 4) + 4 * h32 + v % 4, px, valid)
            # tail: 16 pixels at NB G 128 + 16 p, rows 16 wave .. 16 wave + 15
            px = NB * GP * 128 + 16 * pg + l16
            voff, inside = in_off(px, h16, pend)
            valid = px < pend
            acc16 = np.zeros((16, 16))
            for q in range(nq):
                bv = in_load(voff, 4 * q * cstride, inside)
                av = lds_read(lds, (16 * wave + l16) * pitch + 4 * q + h16)
                Am = np.zeros((16, 4))
                Am[l16, h16] = av
                Bm = np.zeros((4, 16))
                Bm[h16, l16] = bv
                acc16 += Am @ Bm
            for v in range(4):
                store(acc16[4 * h16 + v, l16], k0 + 16 * wave + 4 * h16 + v, px, valid)
    return out, written


# ---------------------------------------------------------------------------
# bf16 kernel for C = 32 with shifted pixel-fastest LDS copies and
# transposing reads (conv_bf16_tr_kernel, family 6).

def tr16_b64(M):
    """ds_read_b64_tr_b16 within one 16-lane group, as measured on gfx950:
    source lane s supplies four 16-bit values M[s][0..3]; lane i receives
    R[i][e] = M[4e + i // 4][i % 4]."""
    R = np.empty((16, 4), dtype=M.dtype)
    for i in range(16):
        for e in range(4):
            R[i, e] = M[4 * e + i // 4, i % 4]
    return R


def emulate_bf16_tr(g, In, Ker, wgs=None, out_aligned=True, out_bf16=False):
    """Transposing-read bf16 kernel (family 6): Ker read in 16-byte vectors of
    its natural order and scattered into the LDS image; per thread one In
    group (channel, 8 pixels) on every RPT-th tile row, shifted back at the
    right edge of the image row; operands In x Ker on the MFMA (rows =
    pixels); each wave's tile in NPART parts whose 16-byte (or, for Q % 4 != 0
    or an unaligned Out, 4-byte) stores are checked lane by lane."""
    N, C, K, H, W, R, S, P, Q = (g[x] for x in "N C K H W R S P Q".split())
    _chk(g["family"] == 6 and g["threads"] == 256, "transposing bf16 geometry")
    TR, TW = g["max_ni"], g["max_nk"]
    _chk(g["tr"] == TR and g["tw"] == TW and C == 32 and K <= 64 and W % 2 == 0 and W >= 8
         and P % TR == 0, "tile")
    RS = R * S
    IN_ROWS = TR + R - 1
    CP = g["in_cstride"]
    _chk(g["in_rows"] == IN_ROWS and CP >= IN_ROWS * TW and CP % 64 == 16, "LDS In planes")
    kpitch = g["ker_rstride"]
    _chk(kpitch == (RS if RS % 2 else RS + 1), "Ker pitch")
    ker_bytes_lds = 64 * kpitch * 64
    lds_bytes = ker_bytes_lds + S * 32 * CP * 2
    _chk(lds_bytes == g["stage_elems"] == g["lds_bytes"] and lds_bytes <= 160 * 1024, "LDS bytes")
    CBR = TW // 16
    WP = TR * CBR // 4
    _chk(g["wp"] == WP and TR * CBR == 4 * WP, "blocks per wave")
    NPART = 2 if WP % 2 == 0 else 1
    PB = WP // NPART
    GPR = TW // 8
    TPR = 32 * GPR
    _chk(256 % TPR == 0, "whole rows per pass")
    RPT = 256 // TPR
    NIT = -(-IN_ROWS // RPT)
    in_size, out_size = N * C * H * W, N * K * P * Q
    _chk(In.size == in_size and Ker.size == K * C * RS and g["in_bytes"] == in_size * 2
         and g["ker_bytes"] == K * C * RS * 2, "sizes")
    _chk(out_size * 4 < 2 ** 31 and in_size * 2 < 2 ** 31, "32-bit buffer offsets")
    OOB = 0x80000000
    vec_out = Q % 4 == 0 and out_aligned  # 16-byte (8-byte for bf16 Out) stores of 4 pixels
    out_e = 2 if out_bf16 else 4
    out = np.full(out_size, np.nan)
    written = np.zeros(out_size, np.int64)
    tiles = g["tiles_rows"] * g["tiles_cols"]
    G = g["grid"]
    # Ker: thread t, vector i covers elements 8v .. 8v+7 (v = t + 256 i) of
    # the natural order (rows past K lie past the buffer and read zeros); the
    # vectors go to the In region in that order, then thread items
    # (kl, tap, octet) gather their eight channels into one 16-byte chunk.
    KV = 64 * 32 * RS // 8
    _chk(KV % 256 == 0 and 64 * 32 * RS * 2 <= S * 32 * CP * 2, "Ker staging")
    raw = np.full(S * 32 * CP, np.nan)
    for v in range(KV):
        off = 16 * v
        _chk(off + 16 <= g["ker_bytes"] or off >= g["ker_bytes"], "Ker vector straddles the end")
        raw[8 * v: 8 * v + 8] = Ker[8 * v: 8 * v + 8] if off + 16 <= g["ker_bytes"] else 0.0
    lker = {}
    for it in range(64 * RS * 4):
        o, rest = it & 3, it >> 2
        rs, kl = rest % RS, rest // RS
        src = [(kl * 32 + 8 * o + e) * RS + rs for e in range(8)]
        _chk(min(src) >= 0 and max(src) < 64 * 32 * RS, "Ker gather inside the staged slice")
        chunk = (kl * kpitch + rs) * 64 + (o ^ ((kl >> 1) & 3)) * 16
        _chk(chunk + 16 <= ker_bytes_lds and chunk % 16 == 0, "Ker chunk bounds")
        for e in range(8):
            addr = chunk + 2 * e
            _chk(addr not in lker, "Ker element written twice")
            lker[addr] = raw[src[e]]
    _chk(len(lker) == 64 * RS * 32, "Ker image complete")

    def kval(kl, rs, c):
        return lker[(kl * kpitch + rs) * 64 + ((c >> 3) ^ ((kl >> 1) & 3)) * 16 + (c & 7) * 2]

    for b in (range(G) if wgs is None else wgs):
        G8 = G & ~7
        L = (b & 7) * (G8 >> 3) + (b >> 3) if b < G8 else b
        for T in range(L, tiles, G):  # tiles L, L + G, ...
            ct, rt = T % g["tiles_cols"], T // g["tiles_cols"]
            rho0 = rt * TR
            n, p0 = divmod(rho0, P)
            q0 = ct * TW
            lin = np.full(S * 32 * CP, np.nan)
            for tid in range(256):
                gr, ic, irow0 = tid % GPR, (tid // GPR) % 32, tid // TPR
                x = q0 + 8 * gr
                over = max(0, x + 8 - W)
                sh = over >> 1
                base = (((n * 32 + ic) * H + p0 + irow0) * W + x) * 2
                for i in range(NIT):
                    row = irow0 + RPT * i
                    ok = row < IN_ROWS and x < W
                    off = base + RPT * i * W * 2
                    o16 = off - 2 * over if ok else OOB
                    o4 = off + 16 if ok and x + 8 < W else OOB
                    if ok:
                        rstart = ((n * 32 + ic) * H + p0 + row) * W * 2
                        _chk(over < 8 and rstart <= o16 and o16 + 16 <= rstart + 2 * W, "16-byte load inside the row")
                    if o4 != OOB:
                        _chk(o4 + 4 <= rstart + 2 * W, "4-byte load inside the row")
                    qv = In[o16 // 2: o16 // 2 + 8] if o16 < g["in_bytes"] else np.zeros(8)
                    d4 = In[o4 // 2: o4 // 2 + 2] if o4 < g["in_bytes"] else np.zeros(2)
                    if row >= IN_ROWS:
                        continue
                    qd = [qv[2 * e: 2 * e + 2] for e in range(4)]
                    dw = [qd[e + sh] if e + sh < 4 else np.zeros(2) for e in range(4)] + [d4]
                    px = np.concatenate(dw)  # pixels x .. x+9 (zeros past the row)
                    if ok:
                        for e in range(10):
                            if x + e < W:
                                _chk(px[e] == In[(((n * 32 + ic) * H + p0 + row) * W) + x + e], "edge shift")
                    dst = ic * CP + row * TW + 8 * gr
                    _chk(dst % 8 == 0 and dst + 8 <= 32 * CP, "LDS copy write")
                    for sx in range(S):
                        lin[sx * 32 * CP + dst: sx * 32 * CP + dst + 8] = px[sx:sx + 8]
            for wave in range(4):
                for part in range(NPART):
                    accs = []
                    for bi in range(PB):
                        bb = wave * WP + part * PB + bi
                        brow, bcol = bb // CBR, 16 * (bb % CBR)
                        acc = np.zeros((4, 16, 16))  # [kb][pixel][k]
                        for r in range(R):
                            for sx in range(S):
                                rs = r * S + sx
                                Am = np.zeros((16, 32))  # pixels x channels (transposing reads)
                                for grp in range(4):
                                    for h in range(2):
                                        M = np.zeros((16, 4))
                                        for s_l in range(16):
                                            src = (sx * 32 * CP + (8 * grp + s_l // 4 + 4 * h) * CP
                                                   + (brow + r) * TW + bcol + 4 * (s_l % 4))
                                            _chk(src % 4 == 0 and 0 <= src and src + 4 <= lin.size,
                                                 "transposing read alignment / bounds")
                                            M[s_l] = lin[src:src + 4]
                                        Rr = tr16_b64(M)  # lane i: channels 8*grp + 4h + e of pixel i
                                        for e in range(4):
                                            Am[:, 8 * grp + 4 * h + e] = Rr[:, e]
                                _chk(not np.isnan(Am).any(), "transposing read of an unwritten element")
                                for kb in range(4):
                                    Bm = np.array([[kval(kb * 16 + jj, rs, c) for jj in range(16)] for c in range(32)])
                                    acc[kb] += Am @ Bm
                        accs.append((acc, brow, bcol))
                    paired = out_bf16 and PB % 2 == 0 and CBR % 2 == 0 and Q % 8 == 0 and out_aligned
                    for bi, (acc, brow, bcol) in enumerate(accs):
                        # stores: lane (j, gq) holds k = 16 kb + j, pixels 4 gq .. 4 gq + 3
                        if paired and bi % 2 == 1:
                            continue  # stored with block bi - 1
                        for jj in range(16):
                            for gq in range(4):
                                pbase = ((n * K + jj) * P + p0) * Q + q0 + 4 * gq
                                col = q0 + bcol + 4 * gq
                                for kb in range(4):
                                    k = kb * 16 + jj
                                    if k >= K:
                                        continue
                                    off = pbase + kb * 16 * P * Q + brow * Q + bcol
                                    if paired:
                                        # 8 pixels per lane: even gq block bi, odd gq block bi + 1
                                        acc1, brow1, bcol1 = accs[bi + 1]
                                        _chk(brow1 == brow and bcol1 == bcol + 16, "paired blocks adjacent")
                                        even = gq % 2 == 0
                                        e8 = off if even else off + 12
                                        c8 = col if even else col + 12
                                        if c8 >= Q:
                                            continue
                                        _chk(e8 % 8 == 0 and c8 % 8 == 0 and c8 + 8 <= Q and (e8 + 8) <= out_size,
                                             "16-byte bf16 store")
                                        src_acc = acc if even else acc1
                                        px0 = 4 * gq if even else 4 * (gq - 1)
                                        for t in range(8):
                                            dst = ((n * K + k) * P + p0 + brow) * Q + c8 + t
                                            _chk(e8 + t == dst, "paired store offset")
                                            out[dst] = src_acc[kb, px0 + t, jj]
                                            written[dst] += 1
                                        continue
                                    vals = acc[kb, 4 * gq: 4 * gq + 4, jj]
                                    if vec_out and not out_bf16:
                                        if col >= Q:
                                            continue
                                        _chk(off % 4 == 0 and (off + 4) * out_e <= out_size * out_e, "vector store")
                                        lanes = range(4)
                                    else:
                                        lanes = [v for v in range(4) if col + v < Q]
                                    for v in lanes:
                                        dst = ((n * K + k) * P + p0 + brow) * Q + col + v
                                        _chk(off + v == dst and col + v < Q, "store offset")
                                        out[dst] = vals[v]
                                        written[dst] += 1
    return out, written


def emulate_phase_split(In, Ker, stride, pad):
    """The two rewrite kernels of conv_fwd_ex, element by element (vectorised
    over the flat output index exactly as the kernels decompose it).  In
    [N,C,H,W], Ker [K,C,R,S] numpy arrays -> (Inp, Kp, (N, C', K, H', W', R',
    S', P, Q)).  Every source index is bounds-checked."""
    N, C, H, W = In.shape
    K, _, R, S = Ker.shape
    sh, sw = stride
    ph, pw = pad
    P, Q = (H + 2 * ph - R) // sh + 1, (W + 2 * pw - S) // sw + 1
    na, nb = min(sh, R), min(sw, S)
    Rp, Sp = -(-R // sh), -(-S // sw)
    Hp, Wp = P + Rp - 1, Q + Sp - 1
    Cp = C * na * nb
    # phase_split_kernel
    i = np.arange(N * Cp * Hp * Wp, dtype=np.int64)
    t = i
    x = t % Wp; t = t // Wp
    y = t % Hp; t = t // Hp
    cp = t % Cp
    n = t // Cp
    b, a, c = cp % nb, (cp // nb) % na, cp // (na * nb)
    iy, ix = y * sh + a - ph, x * sw + b - pw
    inside = (iy >= 0) & (iy < H) & (ix >= 0) & (ix < W)
    src = ((n * C + c) * H + iy) * W + ix
    _chk(np.all((src[inside] >= 0) & (src[inside] < In.size)), "phase split source inside In")
    flat = In.reshape(-1)
    Inp = np.where(inside, flat[np.where(inside, src, 0)], 0.0).reshape(N, Cp, Hp, Wp)
    # ker_phase_kernel
    i = np.arange(K * Cp * Rp * Sp, dtype=np.int64)
    t = i
    tt = t % Sp; t = t // Sp
    rr = t % Rp; t = t // Rp
    cp = t % Cp
    k = t // Cp
    b, a, c = cp % nb, (cp // nb) % na, cp // (na * nb)
    r, s = rr * sh + a, tt * sw + b
    inside = (r < R) & (s < S)
    src = ((k * C + c) * R + r) * S + s
    _chk(np.all((src[inside] >= 0) & (src[inside] < Ker.size)), "Ker rewrite source inside Ker")
    Kp = np.where(inside, Ker.reshape(-1)[np.where(inside, src, 0)], 0.0).reshape(K, Cp, Rp, Sp)
    return Inp, Kp, (N, Cp, K, Hp, Wp, Rp, Sp, P, Q)
