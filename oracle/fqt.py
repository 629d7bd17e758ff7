"""Oracle for the 1-bit FQT layer backward.  TEST INFRASTRUCTURE ONLY.

A plain CPU restatement, step by step and in the paper's order, of what the
backward pass of a binary linear or convolution layer computes under 1-bit
fully quantized training with Activation Gradient Pruning (AGP) and
Sample-Channel joint Quantization (SCQ):

  1. sign binarizer of activations and weights (Section 5.1);
  2. per-group range R and zero point Z of the output gradient, per sample
     (PSQ groups) and per channel (PCQ groups) (Section 3.2; Section 5.2; Section 5.3);
  3. AGP keep probabilities p_i proportional to R_i with sum G/b, Bernoulli masks,
     and the 1/p rescale folded into scale and offset (Section 5.2, the AGP
     definition; Appendix B.2);
  4. b-bit min-max stochastic rounding of every element of a kept group
     (Section 3.2; Proposition B.1);
  5. lossless bit-plane decomposition q = sum_k 2^k q^(k) and LSB-first packing
     (Section 5.2, decomposition; Appendix C, Row_Encoder);
  6. the two integer contractions, dW from PCQ codes and sign(X), dX from PSQ codes
     and sign(W) (Section 5.3, SCQ; Appendix C, Alg. 1 backward);
  7. dequantization by the per-group scales and zero points, and the folder
     that returns the unfolded conv gradient to N x C x H x W (Appendix C,
     {0,1} <-> {+-1} conversion, Unfolder and Folder).

Floating point: the decisions that produce integers (ranges, codes) are taken
in float32 because the paper's kernels quantize float32 gradients and the GPU
takes the same decisions in float32; scale and offset are formed in float64
and stored as float32; the rescaled gradients are produced in float64.
Integer contractions go through a float64 matrix product, which is exact
because every partial sum stays far below 2^53 (asserted).

Where the paper is silent or garbled, the reading taken is stated at the
function.  The functions with no independent pin say "parity unpinned" in their
docstring.
"""
import math
from dataclasses import dataclass, field

import numpy as np

from . import philox

F32 = np.float32
AGP_BERNOULLI, AGP_TOPK, AGP_OFF = 0, 1, 2
WEIGHT_FRACTION_BITS = 40          # fixed-point resolution of the AGP weights (our reading)


# --------------------------------------------------------------------------- shapes

def as_nchw(a):
    """View a linear-layer tensor [N][F] as [N][F][1][1]; 4-D tensors pass through."""
    a = np.asarray(a)
    if a.ndim == 2:
        return a.reshape(a.shape[0], a.shape[1], 1, 1)
    if a.ndim != 4:
        raise ValueError("expected a 2-D (linear) or 4-D (conv) tensor")
    return a


def conv_out_hw(H, W, kh, kw, stride, pad):
    sh, sw = stride
    ph, pw = pad
    return (H + 2 * ph - kh) // sh + 1, (W + 2 * pw - kw) // sw + 1


def canonical_f32(x):
    """float32 copy with -0.0 replaced by +0.0 (reading: a zero point of zero is +0)."""
    return np.asarray(x, dtype=F32) + F32(0.0)


# --------------------------------------------------------------------------- step 1: sign

def sign_bits(x):
    """Bit of the deterministic binarizer (Section 5.1): sign(x) = -1 if x <= 0 else +1.

    Returns the {0,1} bit (1 <=> +1), the form the row encoder of Appendix C
    stores (s = (H > 0)).  NaN compares false and so maps to -1 as well.
    """
    return np.asarray(x) > 0


# --------------------------------------------------------------------------- step 2: ranges

@dataclass
class GroupStats:
    R_s: np.ndarray   # float32 [N] range of each sample's gradient
    Z_s: np.ndarray   # float32 [N] zero point (minimum) of each sample
    R_c: np.ndarray   # float32 [D] range of each channel's gradient
    Z_c: np.ndarray   # float32 [D] zero point of each channel


def group_stats(dy4):
    """Per-group range and zero point (Section 3.2: R = max - min, Z = min;
    Section 5.2 per-sample groups; Section 5.3 per-channel groups).

    dy4 : float32 [N][D][Ho][Wo].  A sample group holds all D*Ho*Wo values of
    sample n; a channel group all N*Ho*Wo values of channel d (reading for
    convolutions: the paper defines PSQ/PCQ on N x D matrices; a conv sample is
    one whole sample, a conv channel one whole output channel).
    R is the float32 difference max - min; Z is the float32 minimum.
    """
    x = canonical_f32(dy4)
    smin, smax = x.min(axis=(1, 2, 3)), x.max(axis=(1, 2, 3))
    cmin, cmax = x.min(axis=(0, 2, 3)), x.max(axis=(0, 2, 3))
    return GroupStats(R_s=(smax - smin) + F32(0.0), Z_s=smin,
                      R_c=(cmax - cmin) + F32(0.0), Z_c=cmin)


# --------------------------------------------------------------------------- step 3: AGP

@dataclass
class AgpResult:
    keep: np.ndarray        # bool [G] mask m_i
    prob: np.ndarray        # float32 [G] keep probability p_i
    scale: np.ndarray       # float32 [G] S_i = R_i / (B p_i) for kept groups, 0 for pruned
    offset: np.ndarray      # float32 [G] Z'_i = Z_i / p_i for kept groups, 0 for pruned
    kept_ids: np.ndarray    # int32 [G] kept ids ascending, then pruned ids ascending
    count: int              # number of kept groups
    weights: list = field(default_factory=list)   # fixed-point weights w_i
    saturated: int = 0      # number of groups whose probability was capped at 1
    w_rem: int = 0          # sum of the weights of the unsaturated groups


def agp_weights(R):
    """Fixed-point AGP weights w_i = floor(2^40 * R_i / R_max) (reading of p_i proportional to R_i).

    The paper writes p_i = N R_i / (b R_total) (Section 5.2).  We keep exact
    proportionality to 2^-40 relative resolution with integer weights, so the
    sum R_total has no summation-order dependence.  R_i / R_max is one correctly
    rounded float64 division.  R_max = 0 gives all-zero weights.
    """
    R = [float(r) for r in np.asarray(R, dtype=F32)]
    rmax = max(R) if R else 0.0
    if rmax <= 0.0:
        return [0] * len(R)
    return [int(math.floor(math.ldexp(r / rmax, WEIGHT_FRACTION_BITS))) for r in R]


def descending_order(w):
    """Group ids sorted by weight, larger first, lower id first among equals."""
    return sorted(range(len(w)), key=lambda i: (-w[i], i))


def water_fill(w, bits):
    """Probabilities with sum G/b, proportional to w, capped at 1 (Section 5.2, AGP).

    The paper's p_i = G R_i / (b R_total) can exceed 1 when one group dominates;
    it is silent on that case.  Reading: cap such groups at p = 1 ("saturate")
    and share the remaining budget G/b - s over the others in proportion to w
    (sampling with probability proportional to size, with certainty units).
    Walking the groups in descending order, group (s) saturates while
    (G - b s) w_(s) >= b W_rem(s), W_rem(s) being the weight of the groups not
    yet saturated.  The unsaturated groups then get p_i = (G - b s) w_i / (b W_rem).
    Returns (order, s, W_rem).
    """
    G, b = len(w), int(bits)
    order = descending_order(w)
    w_rem = sum(w)
    s = 0
    while s < G and w[order[s]] > 0 and (G - b * s) * w[order[s]] >= b * w_rem:
        w_rem -= w[order[s]]
        s += 1
    return order, s, w_rem


def agp_select(R, Z, bits, mode, u32):
    """AGP selection of one group set (Section 5.2; Section 5.3 for the channel set).

    R, Z : float32 [G] ranges and zero points;  u32 : uint32 [G] random words.
    mode : AGP_BERNOULLI -- the paper's m_i ~ Bern(p_i) with p from water_fill;
                           kept iff u32 / 2^32 < p_i, decided exactly in integers:
                           u32 * (b W_rem) < (G - b s) w_i * 2^32.  Saturated groups
                           are always kept.
           AGP_TOPK      -- the deterministic limit p in {1,0} of Appendix B.2: keep the
                           max(1, floor(G/b)) largest weights, p = 1 (biased; an option).
           AGP_OFF       -- plain b-bit PSQ/PCQ, every group kept with p = 1.
    The mask matrix M = diag(m_i / p_i) is folded into the dequantization:
    a kept group's scale is S_i = R_i / (B p_i) and its offset Z'_i = Z_i / p_i
    (scaling a group by 1/p scales its range and zero point alike, so the codes
    of M*grad equal those of grad).  Pruned groups get S = Z' = 0.
    """
    R = np.asarray(R, dtype=F32)
    Z = np.asarray(Z, dtype=F32)
    G, b = R.size, int(bits)
    B = (1 << b) - 1
    keep = np.zeros(G, dtype=bool)
    prob = np.zeros(G, dtype=F32)
    scale = np.zeros(G, dtype=F32)
    offset = np.zeros(G, dtype=F32)
    w = agp_weights(R)
    s, w_rem = 0, sum(w)

    if mode == AGP_OFF:
        keep[:] = True
        prob[:] = 1.0
    elif mode == AGP_TOPK:
        order = descending_order(w)
        k = max(1, G // b)
        for i in order[:k]:
            keep[i] = True
            prob[i] = 1.0
    elif mode == AGP_BERNOULLI:
        order, s, w_rem = water_fill(w, b)
        A = G - b * s
        for i in order[:s]:
            keep[i] = True
            prob[i] = 1.0
        for i in order[s:]:
            if w_rem > 0 and A > 0:
                prob[i] = F32(float(A * w[i]) / float(b * w_rem))
                if w[i] > 0 and int(u32[i]) * (b * w_rem) < A * w[i] * (1 << 32):
                    keep[i] = True
    else:
        raise ValueError("unknown AGP mode")

    saturated_ids = set(descending_order(w)[:s]) if mode == AGP_BERNOULLI else set()
    for i in range(G):
        if not keep[i]:
            continue
        if mode != AGP_BERNOULLI or i in saturated_ids:          # p_i = 1
            scale[i] = F32(float(R[i]) / float(B))
            offset[i] = Z[i]
        else:                                                   # p_i = A w_i / (b W_rem)
            A = G - b * s
            scale[i] = F32((float(R[i]) * float(b * w_rem)) / (float(B) * float(A * w[i])))
            offset[i] = F32((float(Z[i]) * float(b * w_rem)) / float(A * w[i]))
    kept = np.flatnonzero(keep)
    pruned = np.flatnonzero(~keep)
    return AgpResult(keep=keep, prob=prob, scale=scale, offset=offset + F32(0.0),
                     kept_ids=np.concatenate([kept, pruned]).astype(np.int32),
                     count=int(kept.size), weights=w, saturated=s, w_rem=w_rem)


# --------------------------------------------------------------------------- step 4: SR

def sr_codes(x, Z, R, bits, u32):
    """b-bit min-max stochastic rounding (Section 3.2; Proposition B.1).

    q = SR(B (x - Z) / R) with B = 2^b - 1.  Taken in float32, in this order:
    inv = B / R (one correctly rounded division per group), v = (x - Z) * inv
    (two roundings, no fused multiply-add), v clamped to [0, B], then
    q = floor(v) + [u24 < frac(v) * 2^24] with u24 = u32 >> 8, so q rounds up
    with probability frac(v) up to 2^-24 (reading: a 24-bit uniform and a
    strict comparison; an integral v never rounds up).  R = 0 gives q = 0.
    x, Z, R, u32 broadcast against each other.  Returns uint8 codes.
    """
    B = F32((1 << int(bits)) - 1)
    x = np.asarray(x, dtype=F32)
    Z = np.asarray(Z, dtype=F32)
    R = np.asarray(R, dtype=F32)
    safe_R = np.where(R > 0, R, F32(1.0))
    inv = (B / safe_R).astype(F32)
    v = ((x - Z).astype(F32) * inv).astype(F32)
    v = np.minimum(np.maximum(v, F32(0.0)), B)
    fl = np.floor(v)
    frac = (v - fl).astype(F32)
    u24 = (np.asarray(u32, dtype=np.uint32) >> np.uint32(8)).astype(F32)
    q = fl.astype(np.int64) + (u24 < frac * F32(16777216.0)).astype(np.int64)
    q = np.where(R > 0, q, 0)
    return q.astype(np.uint8)


# --------------------------------------------------------------------------- variance

def agp_probabilities(R, bits, mode):
    """Keep probabilities p_i of AGP in float64 (Section 5.2; water_fill's reading for
    p_i > 1): 1 for saturated groups, (G - b s) w_i / (b W_rem) for the others; every
    group with R > 0 has p = 1 under AGP_OFF; TOPK keeps its k groups with p = 1."""
    R = np.asarray(R, dtype=F32)
    G, b = R.size, int(bits)
    w = agp_weights(R)
    p = np.zeros(G)
    if mode == AGP_OFF:
        p[:] = 1.0
    elif mode == AGP_TOPK:
        p[descending_order(w)[:max(1, G // b)]] = 1.0
    else:
        order, s, w_rem = water_fill(w, b)
        p[order[:s]] = 1.0
        if w_rem > 0:
            for i in order[s:]:
                p[i] = (G - b * s) * w[i] / (b * w_rem)
    return p


def quantizer_variance(dy, bits, mode=AGP_BERNOULLI, groups="samples"):
    """Exact conditional variance, element by element, of the quantized gradient that feeds
    one product: g_hat = (m/p) Q(x), with Q the b-bit min-max stochastic-rounding quantizer
    of the element's group (Section 3.2) and m ~ Bern(p) the AGP mask (Section 5.2).

    groups = "samples" (PSQ, the dX operand) or "channels" (PCQ, the dW operand).  With
    Var_SR = (R/B)^2 f (1 - f), f the fractional part of v = clamp((x - Z) B/R, 0, B) taken
    in float32 as the quantizer takes it (Proposition B.1's variance of SR, scaled by R/B),
    E[g_hat] = x and Var[g_hat] = E[g_hat^2] - x^2 = (Var_SR + x^2)/p - x^2
                                = Var_SR / p + x^2 (1 - p) / p.
    Under AGP_OFF (p = 1) this is plain per-group quantization's Var_SR.  Groups with
    p = 0 (R = 0, never kept; reading of the zero-range case) and the groups TOPK prunes
    contribute 0.  Returns float64 in dy's [N][D][Ho][Wo] layout; the sum over all elements
    is the quantizer variance of Section 4.2 / Appendix B.
    """
    dy4 = canonical_f32(as_nchw(dy))
    st = group_stats(dy4)
    if groups == "samples":
        R, Z = st.R_s, st.Z_s
        bshape = (-1, 1, 1, 1)
    elif groups == "channels":
        R, Z = st.R_c, st.Z_c
        bshape = (1, -1, 1, 1)
    else:
        raise ValueError(groups)
    B = F32((1 << int(bits)) - 1)
    p = agp_probabilities(R, bits, mode).reshape(bshape)
    Rb = R.reshape(bshape)
    safe_R = np.where(Rb > 0, Rb, F32(1.0))
    inv = (B / safe_R).astype(F32)
    v = ((dy4 - Z.reshape(bshape)).astype(F32) * inv).astype(F32)
    v = np.minimum(np.maximum(v, F32(0.0)), B).astype(np.float64)
    f = v - np.floor(v)
    var_sr = np.where(Rb > 0, (Rb.astype(np.float64) / float(B)) ** 2 * f * (1.0 - f), 0.0)
    x = dy4.astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        out = np.where(p > 0, var_sr / p + x * x * (1.0 - p) / p, 0.0)
    return out


# --------------------------------------------------------------------------- step 5: planes

def bit_planes(q, bits):
    """Lossless decomposition q = sum_{k<b} 2^k q^(k) (Section 5.2): plane k is (q >> k) & 1."""
    q = np.asarray(q, dtype=np.uint8)
    return np.stack([(q >> np.uint8(k)) & np.uint8(1) for k in range(int(bits))]).astype(bool)


def pack_words(bits):
    """Row encoder (Appendix C, Alg. 2), read as: bit j of a line goes to bit (j % 64) of
    64-bit word j // 64, least significant bit first; a ragged tail is zero-padded.
    bits : bool [..., L]  ->  uint64 [..., ceil(L / 64)].
    """
    bits = np.asarray(bits, dtype=bool)
    L = bits.shape[-1]
    nw = (L + 63) // 64
    padded = np.zeros(bits.shape[:-1] + (nw * 64,), dtype=np.uint8)
    padded[..., :L] = bits
    by = np.ascontiguousarray(np.packbits(padded, axis=-1, bitorder="little"))
    return by.view("<u8").reshape(bits.shape[:-1] + (nw,))


def unpack_words(words, L):
    """Inverse of pack_words: uint64 [..., nw] -> bool [..., L]."""
    words = np.ascontiguousarray(np.asarray(words, dtype="<u8"))
    by = words.view(np.uint8).reshape(words.shape[:-1] + (words.shape[-1] * 8,))
    return np.unpackbits(by, axis=-1, bitorder="little")[..., :L].astype(bool)


# --------------------------------------------------------------------------- AGP + SCQ

@dataclass
class QGrad:
    bits: int
    stats: GroupStats
    samples: AgpResult            # AGP over samples (feeds PSQ, the dX product)
    channels: AgpResult           # AGP over channels (feeds PCQ, the dW product)
    q_psq: np.ndarray             # uint8 [N][D][Ho][Wo] PSQ codes (0 in pruned samples)
    q_pcq: np.ndarray             # uint8 [N][D][Ho][Wo] PCQ codes (0 in pruned channels)
    psq_rows: np.ndarray          # uint8 [Nk*Ho*Wo][D] codes of kept samples, rows (kept n, ho, wo)
    pcq_rows: np.ndarray          # uint8 [Dk][N*Ho*Wo] codes of kept channels, columns (n, ho, wo)
    psq_planes: np.ndarray        # uint64 [b][Nk*Ho*Wo][ceil(D/64)]
    pcq_planes: np.ndarray        # uint64 [b][Dk][ceil(N*Ho*Wo/64)]
    u_elem: np.ndarray            # uint32 [N][D][Ho][Wo] stochastic-rounding words


def agp_scq_quantize(dy, bits, mode=AGP_BERNOULLI, seed=0, step=0, layer_id=0):
    """AGP + SCQ quantization of an output gradient (Section 5.2, Section 5.3; Appendix C, Alg. 1
    backward: pruner, PSQ/PCQ quantizers, row/column encoders).

    dy : float32 [N][D] (linear) or [N][D][Ho][Wo] (conv).
    Samples are pruned with masks drawn from stream SAMPLE, channels with
    stream CHANNEL; each element draws one word from stream ELEM (its NCHW linear
    index), shared by its PSQ and its PCQ code (reading: the paper treats dX and dW
    separately, each marginal stays unbiased).
    PSQ codes are packed along D for every pixel of a kept sample (row encoder);
    PCQ codes along N*Ho*Wo for every kept channel (column encoder).
    """
    dy4 = canonical_f32(as_nchw(dy))
    N, D, Ho, Wo = dy4.shape
    P = Ho * Wo
    st = group_stats(dy4)
    us = philox.uniform_words(np.arange(N), philox.STREAM_SAMPLE, seed, step, layer_id)
    uc = philox.uniform_words(np.arange(D), philox.STREAM_CHANNEL, seed, step, layer_id)
    samples = agp_select(st.R_s, st.Z_s, bits, mode, us)
    channels = agp_select(st.R_c, st.Z_c, bits, mode, uc)
    ue = philox.uniform_words(np.arange(N * D * P), philox.STREAM_ELEM, seed, step,
                              layer_id).reshape(N, D, Ho, Wo)
    q_psq = sr_codes(dy4, st.Z_s[:, None, None, None], st.R_s[:, None, None, None], bits, ue)
    q_pcq = sr_codes(dy4, st.Z_c[None, :, None, None], st.R_c[None, :, None, None], bits, ue)
    q_psq[~samples.keep] = 0
    q_pcq[:, ~channels.keep] = 0
    ks = samples.kept_ids[:samples.count]
    kc = channels.kept_ids[:channels.count]
    psq_rows = q_psq[ks].transpose(0, 2, 3, 1).reshape(ks.size * P, D)
    pcq_rows = q_pcq[:, kc].transpose(1, 0, 2, 3).reshape(kc.size, N * P)
    return QGrad(bits=int(bits), stats=st, samples=samples, channels=channels,
                 q_psq=q_psq, q_pcq=q_pcq, psq_rows=psq_rows, pcq_rows=pcq_rows,
                 psq_planes=pack_words(bit_planes(psq_rows, bits)),
                 pcq_planes=pack_words(bit_planes(pcq_rows, bits)),
                 u_elem=ue)


# --------------------------------------------------------------------------- signs and unfolding

def unfold_sign_bits(x4, kh, kw, stride=(1, 1), pad=(0, 0)):
    """sign(unfold(X)) as bits (Section 5.1 binarizer; Appendix C, Unfolder).

    x4 : [N][C][H][W].  Returns bool [C*kh*kw][N*Ho*Wo]: row (c, i, j) holds the
    bits X[n, c, ho*sh - ph + i, wo*sw - pw + j] > 0 over columns (n, ho, wo).
    Reading for padding: the unfold is zero-padded and then binarized, so a
    padded position has sign -1 (bit 0).  Parity unpinned only in that reading
    of the paper's silence; the value itself is pinned against a padded torch
    convolution in the tests.
    """
    x4 = np.asarray(x4)
    N, C, H, W = x4.shape
    sh, sw = stride
    ph, pw = pad
    Ho, Wo = conv_out_hw(H, W, kh, kw, stride, pad)
    padded = np.zeros((N, C, H + 2 * ph, W + 2 * pw), dtype=bool)
    padded[:, :, ph:ph + H, pw:pw + W] = sign_bits(x4)
    U = np.empty((C, kh, kw, N, Ho, Wo), dtype=bool)
    for i in range(kh):
        for j in range(kw):
            win = padded[:, :, i:i + sh * (Ho - 1) + 1:sh, j:j + sw * (Wo - 1) + 1:sw]
            U[:, i, j] = win.transpose(1, 0, 2, 3)
    return U.reshape(C * kh * kw, N * Ho * Wo)


def weight_sign_bits(w):
    """sign(Theta) as bits with the unfolded weight Theta_u in R^{D x C k^2} (Appendix C,
    Unfolder), transposed to [C*kh*kw][D] so each row runs along the contraction D."""
    w = np.asarray(w)
    D = w.shape[0]
    return sign_bits(w.reshape(D, -1)).T.copy()


def int_matmul(a, b):
    """Exact integer matrix product of small integer matrices via float64.

    Every term and partial sum is an integer of magnitude below 2^53, so the
    float64 product is exact; this is asserted from the operand bounds.
    """
    a = np.asarray(a, dtype=np.int64)
    b = np.asarray(b, dtype=np.int64)
    if a.size and b.size:
        bound = int(np.abs(a).max()) * int(np.abs(b).max()) * a.shape[-1]
        assert bound < 2 ** 53, "integer product would not be exact in float64"
    return np.rint(a.astype(np.float64) @ b.astype(np.float64)).astype(np.int64)


def fold_add(cols, N, C, H, W, kh, kw, stride=(1, 1), pad=(0, 0)):
    """Folder (Appendix C): scatter-add unfolded rows back to [N][C][H][W].

    cols : [N*Ho*Wo][C*kh*kw] with rows (n, ho, wo) and columns (c, i, j); the
    value at (n, ho, wo, c, i, j) lands on X position (n, c, ho*sh - ph + i,
    wo*sw - pw + j); positions in the padding are dropped.
    """
    sh, sw = stride
    ph, pw = pad
    Ho, Wo = conv_out_hw(H, W, kh, kw, stride, pad)
    c6 = np.asarray(cols).reshape(N, Ho, Wo, C, kh, kw)
    out = np.zeros((N, C, H + 2 * ph, W + 2 * pw), dtype=c6.dtype)
    for i in range(kh):
        for j in range(kw):
            out[:, :, i:i + sh * (Ho - 1) + 1:sh, j:j + sw * (Wo - 1) + 1:sw] += \
                c6[:, :, :, :, i, j].transpose(0, 3, 1, 2)
    return out[:, :, ph:ph + H, pw:pw + W]


# --------------------------------------------------------------------------- steps 6-7: products

@dataclass
class Backward:
    qgrad: QGrad
    xbits: np.ndarray       # bool [C*kh*kw][N*Ho*Wo]  sign bits of unfold(X)
    wbits: np.ndarray       # bool [C*kh*kw][D]        sign bits of Theta_u, transposed
    xsign_colsum: np.ndarray  # int64 [C*kh*kw] sum over the contraction of sign(unfold(X))
    wsign_colsum: np.ndarray  # int64 [C*kh*kw] sum over D of sign(Theta_u)
    I_dw: np.ndarray        # int64 [D][C*kh*kw]   sum_r q_pcq * sign(X_u); 0 in pruned channels
    I_dx: np.ndarray        # int64 [N][C][H][W]   folded sum_d q_psq * sign(Theta); 0 in pruned samples
    c_dx: np.ndarray        # int64 [C][H][W]      folded column sums of sign(Theta_u)
    dW: np.ndarray          # float64 [D][C][kh][kw] (linear: [D][C])
    dX: np.ndarray          # float64 [N][C][H][W]  (linear: [N][C])
    dW_t1: np.ndarray = None  # float64 |S I| terms, for the cancellation-aware tolerance
    dW_t2: np.ndarray = None  # float64 |Z' c| terms
    dX_t1: np.ndarray = None
    dX_t2: np.ndarray = None


def layer_backward(x, w, dy, bits, mode=AGP_BERNOULLI, seed=0, step=0, layer_id=0,
                   stride=(1, 1), pad=(0, 0), dw_channels=None):
    """Backward of a binary linear/conv layer under 1-bit FQT (Section 5.2 Eq. 21 with
    Section 5.3's SCQ form; Appendix C, Alg. 1 backward).

      dX = S_PSQ qbar_PSQ sign(Theta)^T  (+ zero-point term),  per kept sample
      dW = sign(H)^T qbar_PCQ S_PCQ      (+ zero-point term),  per kept channel

    with the {0,1}/{+-1} conversion of Appendix C read as the exact identity
    sum_j (S q_j + Z') s_j = S sum_j q_j s_j + Z' sum_j s_j.  Layouts follow torch:
    x [N][C] or [N][C][H][W], w [D][C] or [D][C][kh][kw], dy [N][D] or [N][D][Ho][Wo];
    dW has w's shape, dX has x's shape (both float64 here).  Pruned channels give
    zero rows of dW and pruned samples zero samples of dX.  The conv dX goes
    through the paper's route: unfolded product, then the folder.

    dw_channels (optional): output-channel ids; dW, I_dw and their terms are then returned
    for those channels only, as [len(dw_channels)][C*kh*kw] rows in that order (for layers
    whose full D x C*kh*kw float64 arrays would not fit a test's budget).
    """
    linear = np.asarray(x).ndim == 2
    x4, w4, dy4 = as_nchw(x), as_nchw(w), as_nchw(dy)
    N, C, H, W = x4.shape
    D, _, kh, kw = w4.shape
    Ho, Wo = conv_out_hw(H, W, kh, kw, stride, pad)
    assert dy4.shape == (N, D, Ho, Wo), "dy shape does not match the layer"
    K = C * kh * kw
    P = Ho * Wo
    qg = agp_scq_quantize(dy4, bits, mode, seed, step, layer_id)
    xbits = unfold_sign_bits(x4, kh, kw, stride, pad)            # [K][N*P]
    wbits = weight_sign_bits(w4)                                  # [K][D]
    sx = xbits.astype(np.int64) * 2 - 1
    sw = wbits.astype(np.int64) * 2 - 1
    cx = sx.sum(axis=1)
    cw = sw.sum(axis=1)

    # dW: PCQ codes of kept channels against sign(unfold(X)), rescaled per channel.
    ch = qg.channels
    rows = np.arange(D) if dw_channels is None else np.asarray(dw_channels, dtype=np.int64)
    slot_of = {int(d): j for j, d in enumerate(ch.kept_ids[:ch.count])}   # row of pcq_rows
    live = np.array([int(d) in slot_of for d in rows], dtype=bool)        # kept channels
    kept_rows = np.array([slot_of[int(d)] for d in rows[live]], dtype=np.int64)
    kd = rows[live]
    I_dw = np.zeros((rows.size, K), dtype=np.int64)
    I_dw[live] = int_matmul(qg.pcq_rows[kept_rows], sx.T)
    dW = np.zeros((rows.size, K), dtype=np.float64)
    t1w = np.zeros((rows.size, K))
    t2w = np.zeros((rows.size, K))
    t1w[live] = ch.scale[kd, None].astype(np.float64) * I_dw[live]
    t2w[live] = ch.offset[kd, None].astype(np.float64) * cx[None, :]
    dW[live] = t1w[live] + t2w[live]

    # dX: PSQ codes of kept samples against sign(Theta), dequantized, unfolded product, fold.
    sm = qg.samples
    ks = sm.kept_ids[:sm.count]
    Nk = ks.size
    I_u = int_matmul(qg.psq_rows, sw.T)                           # [Nk*P][K]
    I_dx = np.zeros((N, C, H, W), dtype=np.int64)
    I_dx[ks] = fold_add(I_u, Nk, C, H, W, kh, kw, stride, pad)
    row_sample = np.repeat(ks, P)
    g_rows = (sm.scale[row_sample, None].astype(np.float64) * qg.psq_rows
              + sm.offset[row_sample, None].astype(np.float64))     # dequantized PSQ gradient rows
    dX = np.zeros((N, C, H, W), dtype=np.float64)
    dX[ks] = fold_add(g_rows @ sw.T.astype(np.float64), Nk, C, H, W, kh, kw, stride, pad)
    c_dx = fold_add(np.repeat(cw[None, :], P, axis=0), 1, C, H, W, kh, kw, stride, pad)[0]
    t1x = np.zeros((N, C, H, W))
    t2x = np.zeros((N, C, H, W))
    t1x[ks] = sm.scale[ks, None, None, None].astype(np.float64) * I_dx[ks]
    t2x[ks] = sm.offset[ks, None, None, None].astype(np.float64) * c_dx[None]

    if dw_channels is None:
        wshape = (D, C) if linear else (D, C, kh, kw)
    else:
        wshape = (rows.size, K)
    xshape = (N, C) if linear else (N, C, H, W)
    return Backward(qgrad=qg, xbits=xbits, wbits=wbits, xsign_colsum=cx, wsign_colsum=cw,
                    I_dw=I_dw, I_dx=I_dx, c_dx=c_dx,
                    dW=dW.reshape(wshape), dX=dX.reshape(xshape),
                    dW_t1=t1w.reshape(wshape), dW_t2=t2w.reshape(wshape),
                    dX_t1=t1x.reshape(xshape), dX_t2=t2x.reshape(xshape))


# --------------------------------------------------------------------------- forward (binary layer)

@dataclass
class Forward:
    I: np.ndarray           # int64 [N][D][Ho][Wo] (linear: [N][D]) sum_k sign(X_u) sign(Theta_u)
    Y: np.ndarray           # float64, I scaled by Gamma per output channel


def layer_forward(x, w, gamma, stride=(1, 1), pad=(0, 0)):
    """Forward of a binary linear/conv layer (Section 5.1: H = (sign(H_prev) sign(Theta))
    scaled per output channel by the learnable Gamma; Appendix C, Alg. 1 forward with the
    Unfolder for convolutions).

    x : [N][C] (linear) or [N][C][H][W];  w : [D][C] or [D][C][kh][kw];  gamma : [D].
    The integer product I[r][d] = sum over k = (c, i, j) of sign(X_u)[r][k] sign(Theta_u)[d][k]
    is exact; Y = gamma_d * I in float64.  Padding as in unfold_sign_bits (sign -1).
    """
    x = np.asarray(x)
    w = np.asarray(w)
    gamma = np.asarray(gamma, dtype=np.float64)
    linear = x.ndim == 2
    x4 = x.reshape(x.shape[0], x.shape[1], 1, 1) if linear else x
    D = w.shape[0]
    kh, kw = (1, 1) if linear else w.shape[2:]
    N, C, H, W = x4.shape
    Ho, Wo = conv_out_hw(H, W, kh, kw, stride, pad)
    sx = unfold_sign_bits(x4, kh, kw, stride, pad).astype(np.int64) * 2 - 1   # [K][R]
    sw = weight_sign_bits(w).astype(np.int64) * 2 - 1                          # [K][D]
    I_rd = int_matmul(sx.T, sw)                                                # [R][D]
    I = I_rd.reshape(N, Ho, Wo, D).transpose(0, 3, 1, 2)
    Y = I.astype(np.float64) * gamma[None, :, None, None]
    if linear:
        I, Y = I.reshape(N, D), Y.reshape(N, D)
    return Forward(I=I, Y=Y)
