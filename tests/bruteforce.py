"""Brute-force scalar decoder for tiny inputs, used to pin the oracle.

Written independently of oracle/: plain Python lists and loops, the ``math``
module, RoPE as multiplication by unit complex numbers, attention with an
explicit visible-key list per query, and the pixel shuffles as per-pixel index
arithmetic. It follows the paper's definitions (Sec. 3.2-3.4, Algorithm 1) for
one stream; it is far too slow for anything but a handful of tokens.
"""
import cmath
import math


def matvec(Wm, b, x):
    """y_o = sum_i Wm[o][i] x_i + b_o with Wm given as nested lists [out][in]."""
    return [sum(Wm[o][i] * x[i] for i in range(len(x))) + b[o] for o in range(len(Wm))]


def norm_vec(cfg, Wd, prefix, x):
    n = len(x)
    g = Wd[prefix + ".g"]
    if cfg.norm_kind == "rms":
        r = math.sqrt(sum(e * e for e in x) / n + cfg.norm_eps)
        return [x[i] / r * g[i] for i in range(n)]
    mu = sum(x) / n
    var = sum((e - mu) ** 2 for e in x) / n
    b = Wd[prefix + ".b"]
    return [(x[i] - mu) / math.sqrt(var + cfg.norm_eps) * g[i] + b[i] for i in range(n)]


def rms_vec(x, g, eps):
    r = math.sqrt(sum(e * e for e in x) / len(x) + eps)
    return [x[i] / r * g[i] for i in range(len(x))]


def rope_vec(x, pos, theta):
    """Rotate pairs of x (one head) as complex numbers; sections (Dh/4, 3Dh/8, 3Dh/8)."""
    dh = len(x)
    sizes = [dh // 4, (3 * dh) // 8]
    sizes.append(dh - sizes[0] - sizes[1])
    out = list(x)
    off = 0
    for axis in range(3):
        d = sizes[axis]
        for i in range(d // 2):
            ang = pos[axis] * theta ** (-2.0 * i / d)
            zc = complex(x[off + 2 * i], x[off + 2 * i + 1]) * cmath.exp(1j * ang)
            out[off + 2 * i] = zc.real
            out[off + 2 * i + 1] = zc.imag
        off += d
    return out


def _lists(W):
    out = {}
    for k, v in W.items():
        out[k] = v.tolist()
    return out


def decode(cfg, W, z):
    """Decode one stream z [C'][T'][H'][W'] (numpy or nested lists) in full.

    Returns nested lists pixels[c][frame][y][x] (frames = T' r_t).
    """
    Wd = _lists(W)
    zl = z.tolist() if hasattr(z, "tolist") else z
    Cp, T = len(zl), len(zl[0])
    p, Ht, Wt = cfg.patch, cfg.grid_h, cfg.grid_w
    L = Ht * Wt
    D, N, G, Dh = cfg.dim, cfg.n_heads, cfg.n_kv_groups, cfg.head_dim
    r, s, C = cfg.r_t, cfg.s_out, cfg.out_channels

    # token list of one stack: dicts with frame index (latent), temporal pos, h, w
    def embed_tokens():
        toks = []
        for t in range(T):
            for h in range(Ht):
                for w in range(Wt):
                    u = []
                    for c in range(Cp):
                        for i in range(p):
                            for j in range(p):
                                u.append(zl[c][t][p * h + i][p * w + j])
                    x = matvec(Wd["embed.w"], Wd["embed.b"], u)
                    toks.append({"frame": t, "tau": t, "h": h, "w": w, "x": x})
        return toks

    def visible(qt, kt):
        uq = qt["frame"] // cfg.unit_frames
        uk = kt["frame"] // cfg.unit_frames
        return uq - cfg.window < uk <= uq

    def run_stack(name, toks, nblk):
        for bi in range(nblk):
            pf = f"{name}.{bi}"
            qs, ks, vs = [], [], []
            for tk in toks:
                a = norm_vec(cfg, Wd, pf + ".norm1", tk["x"])
                y = matvec(Wd[pf + ".wqkv"], Wd[pf + ".bqkv"], a)
                q = [y[n * Dh:(n + 1) * Dh] for n in range(N)]
                k = [y[D + g * Dh:D + (g + 1) * Dh] for g in range(G)]
                v = [y[D + G * Dh + g * Dh:D + G * Dh + (g + 1) * Dh] for g in range(G)]
                if cfg.kv_norm:
                    k = [rms_vec(e, Wd[pf + ".knorm.g"], cfg.norm_eps) for e in k]
                    v = [rms_vec(e, Wd[pf + ".vnorm.g"], cfg.norm_eps) for e in v]
                if cfg.rope:
                    pos = (tk["tau"], tk["h"], tk["w"])
                    q = [rope_vec(e, pos, cfg.rope_theta) for e in q]
                    k = [rope_vec(e, pos, cfg.rope_theta) for e in k]
                qs.append(q)
                ks.append(k)
                vs.append(v)
            new_x = []
            for qi, tq in enumerate(toks):
                keys = [ki for ki, tk in enumerate(toks) if visible(tq, tk)]
                o = []
                for n in range(N):
                    g = (n * G) // N
                    sc = [sum(qs[qi][n][d] * ks[ki][g][d] for d in range(Dh)) / math.sqrt(Dh)
                          for ki in keys]
                    mx = max(sc)
                    e = [math.exp(v_ - mx) for v_ in sc]
                    tot = sum(e)
                    for d in range(Dh):
                        o.append(sum(e[j] * vs[keys[j]][g][d] for j in range(len(keys))) / tot)
                x = tq["x"]
                ao = matvec(Wd[pf + ".wo"], Wd[pf + ".bo"], o)
                x = [x[i] + ao[i] for i in range(D)]
                a = norm_vec(cfg, Wd, pf + ".norm2", x)
                if cfg.mlp_kind == "swiglu":
                    H = cfg.mlp_hidden
                    gu = matvec(Wd[pf + ".w13"], Wd[pf + ".b13"], a)
                    hid = [gu[i] / (1.0 + math.exp(-gu[i])) * gu[H + i] for i in range(H)]
                else:
                    pre = matvec(Wd[pf + ".w1"], Wd[pf + ".b1"], a)
                    hid = [0.5 * e * (1.0 + math.erf(e / math.sqrt(2.0))) for e in pre]
                m = matvec(Wd[pf + ".w2"], Wd[pf + ".b2"], hid)
                new_x.append([x[i] + m[i] for i in range(D)])
            for tk, x in zip(toks, new_x):
                tk["x"] = x
        for tk in toks:
            tk["y"] = norm_vec(cfg, Wd, name + ".norm_f", tk["x"])
        return toks

    toks = run_stack("bb", embed_tokens(), cfg.n_backbone_blocks)
    # per output frame fo and token (h, w): feature vector of C s^2 channels
    feats = {}
    if cfg.head_kind == "temporal_first":
        rtoks = []
        for t in range(T):
            for j in range(r):
                for tk in toks:
                    if tk["frame"] != t:
                        continue
                    tt = matvec(Wd["tup.w"], Wd["tup.b"], tk["y"])
                    rtoks.append({"frame": t, "tau": r * t + j, "sub": j, "h": tk["h"],
                                  "w": tk["w"], "x": tt[j * D:(j + 1) * D]})
        rtoks = run_stack("rf", rtoks, cfg.n_refine_blocks)
        for tk in rtoks:
            hid = matvec(Wd["head1.w"], Wd["head1.b"], tk["y"])
            hid = [e / (1.0 + math.exp(-e)) for e in hid]
            feats[(tk["frame"] * r + tk["sub"], tk["h"], tk["w"])] = \
                matvec(Wd["head2.w"], Wd["head2.b"], hid)
    else:
        for tk in toks:
            f = matvec(Wd["head.w"], Wd["head.b"], tk["y"])
            for j in range(r):
                feats[(tk["frame"] * r + j, tk["h"], tk["w"])] = \
                    f[j * C * s * s:(j + 1) * C * s * s]
    pix = [[[[0.0] * (Wt * s) for _ in range(Ht * s)] for _ in range(T * r)] for _ in range(C)]
    for c in range(C):
        for fo in range(T * r):
            for yy in range(Ht * s):
                for xx in range(Wt * s):
                    f = feats[(fo, yy // s, xx // s)]
                    v_ = f[c * s * s + (yy % s) * s + (xx % s)]
                    if cfg.clamp_output:
                        v_ = min(1.0, max(-1.0, v_))
                    pix[c][fo][yy][xx] = v_
    return pix


# --------------------------------------------------------------------------
# FP8 (E4M3) MLP of the "-Opt" decoder (Sec. 4.6), scalar form. Roundings come
# from struct (IEEE single and half, round to nearest even) and from a search
# over the E4M3 code table built from its bit fields.
# --------------------------------------------------------------------------
import struct


def f32(x):
    return struct.unpack("f", struct.pack("f", x))[0]


def f16(x):
    return struct.unpack("e", struct.pack("e", x))[0]


def _e4m3_table():
    out = []
    for sgn in (1.0, -1.0):
        for e in range(16):
            for m in range(8):
                if e == 15 and m == 7:      # NaN code
                    continue
                v = (m / 8.0) * 2.0 ** -6 if e == 0 else (1.0 + m / 8.0) * 2.0 ** (e - 7)
                out.append((sgn * v, m))
    return out


_E4M3 = _e4m3_table()


def e4m3_nearest(x):
    """Nearest finite E4M3 value; at a midpoint the one with an even mantissa
    field; beyond +-448 the largest value of that sign."""
    if x >= 448.0:
        return 448.0
    if x <= -448.0:
        return -448.0
    best, bm, bd = None, None, None
    for v, m in _E4M3:
        d = abs(v - x)
        if bd is None or d < bd or (d == bd and m % 2 == 0 and bm % 2 == 1):
            best, bm, bd = v, m, d
    return best + 0.0


def quant_row(row, amax=None):
    """E4M3 codes (as values) and scale of one row: per row (amax None) with
    m = max |fp32(x)|, else at the fixed amplitude amax; inv = fp32(448 / m),
    code = e4m3(fp32(fp32(x) inv)), scale = fp32(m / 448); a zero row takes m = 448."""
    x32 = [f32(v) for v in row]
    m = f32(amax) if amax is not None else max(abs(v) for v in x32)
    if m == 0.0:
        m = 448.0
    inv = f32(448.0 / m)
    return [e4m3_nearest(f32(v * inv)) for v in x32], f32(m / 448.0)


def fp8_linear_rows(rows, Wm, b, amax=None):
    """y = x W^T + b with the rows of x quantised per row (or at amax) and the
    rows of W per output channel: sum of code products times both scales."""
    qw = [quant_row(w) for w in Wm]
    out = []
    for r in rows:
        cx, sx = quant_row(r, amax)
        out.append([sum(cx[k] * cw[k] for k in range(len(cx))) * sx * sw + b[n]
                    for n, (cw, sw) in enumerate(qw)])
    return out


def fp8_mlp(cfg, W, p, rows, mode):
    """The SwiGLU MLP of block p on the given input rows with both GEMMs on
    E4M3 operands; the SwiGLU output is held in fp16 between them. mode "fp8":
    activations quantised per row; "fp8s": at the block's fixed amplitudes
    W[p + ".amax_in"], W[p + ".amax_hid"]."""
    H = cfg.mlp_hidden
    Wd = {k: W[k].tolist() for k in (p + ".w13", p + ".b13", p + ".w2", p + ".b2")}
    a_in = float(W[p + ".amax_in"]) if mode == "fp8s" else None
    a_hid = float(W[p + ".amax_hid"]) if mode == "fp8s" else None
    y = fp8_linear_rows(rows, Wd[p + ".w13"], Wd[p + ".b13"], a_in)
    hid = [[f16(r[i] / (1.0 + math.exp(-r[i])) * r[H + i]) for i in range(H)] for r in y]
    return fp8_linear_rows(hid, Wd[p + ".w2"], Wd[p + ".b2"], a_hid)
