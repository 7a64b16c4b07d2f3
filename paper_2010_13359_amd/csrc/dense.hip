// Element-major kernels of Algorithm 2 (arXiv:2010.13359): the statistics
// pass of the segment-scaled compressors (scaled sign, s-level quantizer,
// m-bit sign-magnitude quantizer), the fused apply pass of every compressor
// (top-k included), and the separate pack / unpack / aggregate / OMD kernels.
//
// Passes over HBM per iteration:
//   1. segment statistics: per (worker, segment) sum |p|, sum p^2 or max |p|
//      of p = fl(fl(eta g) + e), one workgroup per piece, binary64 partials;
//      a tiny kernel then combines the partials of each segment in piece
//      order (deterministic) into the scale and the quantizer constants.
//   2. the fused apply pass (k_fused_split): a workgroup covers 256 elements
//      of all M workers, its waves splitting the workers; each lane encodes
//      one quad of 4 elements per worker row, writes e_t and the message,
//      keeps p-hat and fl(eta g) + e_t in registers; the ascending-worker sum
//      is chained through LDS; the last wave of the chain applies
//      w_t = w_{t-1} - q-hat; every wave then writes its rows' evaluation
//      points w_t - (fl(eta g) + e_t).  k_fused (one lane walks all M rows)
//      serves M > 128.
#include <type_traits>

#include "device.hpp"
#include "plan.hpp"

namespace dq {

namespace {

enum { kSign = DQGAN_SIGN, kQsgd = DQGAN_QSGD, kTopk = DQGAN_TOPK, kIdentity = DQGAN_IDENTITY, kMbit = DQGAN_MBIT };

// ---------------------------------------------------------------------------
// Pass 1: segment statistics.

template <int NORM>
__global__ __launch_bounds__(kBlock) void k_segment_partials(const float *__restrict__ G, const float *__restrict__ E,
                                                             float eta, int64_t ld, const Piece *__restrict__ pieces,
                                                             int32_t n_pieces, double *__restrict__ partial,
                                                             float *__restrict__ pmax) {
    const int pc = blockIdx.x;
    const int m = blockIdx.y;
    const Piece P = pieces[pc];
    const float *g = G + static_cast<int64_t>(m) * ld;
    const float *e = E + static_cast<int64_t>(m) * ld;
    const int64_t lo = P.start, hi = P.start + P.len;
    const int64_t q0 = lo >> 2, q1 = (hi + 3) >> 2;
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    float mx = 0.0f;
    // Four quads per thread per trip, all eight loads issued before use.
    constexpr int U = 4;
    for (int64_t qb = q0 + threadIdx.x; qb < q1; qb += U * kBlock) {
        f32x4 gv[U], ev[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t q = qb + u * kBlock;
            if (q < q1) {
                gv[u] = ld_stream(g + 4 * q);
                ev[u] = ld_stream(e + 4 * q);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t q = qb + u * kBlock;
            if (q >= q1) break;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int64_t i = 4 * q + c;
                const float p = add_rn(mul_rn(eta, elem(gv[u], c)), elem(ev[u], c));
                const bool in = (i >= lo) && (i < hi);
                if (NORM == DQGAN_L1) {
                    acc[c] += in ? static_cast<double>(fabsf(p)) : 0.0;
                } else if (NORM == DQGAN_L2) {
                    const double pd = static_cast<double>(p);
                    acc[c] += in ? pd * pd : 0.0;  // the product is exact in binary64
                } else {
                    mx = in ? fmaxf(mx, fabsf(p)) : mx;
                }
            }
        }
    }
    __shared__ double sh[kBlock / 64];
    __shared__ float shm[kBlock / 64];
    double s = (acc[0] + acc[1]) + (acc[2] + acc[3]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        s += __shfl_xor(s, o);
        mx = fmaxf(mx, __shfl_xor(mx, o));
    }
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
        sh[wave] = s;
        shm[wave] = mx;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        const int64_t o = static_cast<int64_t>(m) * n_pieces + pc;
        partial[o] = (sh[0] + sh[1]) + (sh[2] + sh[3]);
        pmax[o] = fmaxf(fmaxf(shm[0], shm[1]), fmaxf(shm[2], shm[3]));
    }
}

// Combine the partials of each (worker, segment) in piece order, or take the
// caller's scales, and derive the per-segment constants (SegConst): SIGN the
// scale; QSGD, MBIT fl(s/(u sigma)) and fl(u sigma/s), negated when u = 2^64
// (sigma < 2^-64), zeros for sigma = 0 or not finite.  Quotients of two
// binary32 values computed in binary64 and rounded to binary32 equal the
// correctly rounded binary32 quotient (53 >= 2*24 + 2).
__global__ __launch_bounds__(kBlock) void k_finalize(int kind, int norm, int levels, const double *__restrict__ partial,
                                                     const float *__restrict__ pmax, int32_t n_pieces,
                                                     const int32_t *__restrict__ seg_piece,
                                                     const int64_t *__restrict__ off, int32_t M, int32_t n_seg,
                                                     const float *__restrict__ scales_in, float *__restrict__ scale_out,
                                                     SegConst *__restrict__ consts) {
    // One wave per (worker, segment): lane l adds the segment's pieces
    // l, l+64, ... in order, then a fixed butterfly combines the lanes.
    const int64_t tid = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) >> 6;
    const int lane = threadIdx.x & 63;
    if (tid >= static_cast<int64_t>(M) * n_seg) return;
    const int m = static_cast<int>(tid / n_seg);
    const int j = static_cast<int>(tid % n_seg);
    float sc;
    if (scales_in) {
        sc = scales_in[tid];
    } else if (norm == DQGAN_LINF) {
        float mx = 0.0f;
        for (int p = seg_piece[j] + lane; p < seg_piece[j + 1]; p += 64)
            mx = fmaxf(mx, pmax[static_cast<int64_t>(m) * n_pieces + p]);
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
        sc = mx;
    } else {
        double s = 0.0;
        for (int p = seg_piece[j] + lane; p < seg_piece[j + 1]; p += 64)
            s += partial[static_cast<int64_t>(m) * n_pieces + p];
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
        if (norm == DQGAN_L1)
            sc = static_cast<float>(s / static_cast<double>(off[j + 1] - off[j]));
        else
            sc = static_cast<float>(sqrt(s));
    }
    if (lane != 0) return;
    if (scale_out) scale_out[tid] = sc;
    SegConst c{sc, 0.0f};
    if (kind == kQsgd || kind == kMbit) {
        c.a = 0.0f;
        if (sc > 0.0f && sc <= 3.402823466e38f) {
            const bool tiny = sc < 0x1.0p-64f;
            // u * sigma is exact: a power of two times a binary32 value
            const double sd = static_cast<double>(sc) * (tiny ? 0x1.0p64 : 1.0), lv = static_cast<double>(levels);
            c.a = static_cast<float>(lv / sd);
            c.b = static_cast<float>(sd / lv);
            if (tiny) {
                c.a = -c.a;
                c.b = -c.b;
            }
        }
    }
    consts[tid] = c;
}

// r = fl(|p| s / sigma) of equation (qsgd) from the constant a of SegConst
// (negative: |p| is first multiplied by 2^64), and the decoded magnitude
// fl(level sigma / s) from its constant b (negative: multiplied back by
// 2^-64).  The extra products are exact or the one final rounding.
__device__ __forceinline__ float level_ratio(float abs_p, float ca) {
    return mul_rn(mul_rn(abs_p, ca < 0.0f ? 0x1.0p64f : 1.0f), fabsf(ca));
}
__device__ __forceinline__ float level_magnitude(uint32_t level, float cb) {
    return mul_rn(mul_rn(static_cast<float>(level), fabsf(cb)), cb < 0.0f ? 0x1.0p-64f : 1.0f);
}

// ---------------------------------------------------------------------------
// Per-quad encode of one worker row (shared by the row kernel and the fused
// step).  Outputs: eg = fl(eta g), p-hat, e_t = fl(p - p-hat), the 4 sign bits
// and the 4 level fields (8 bits each, packed low to high).

struct QuadCodes {
    f32x4 eg, phat, enew;
    uint32_t sign_nib;
    uint32_t levels;
};

template <int KIND>
__device__ __forceinline__ QuadCodes encode_quad(const f32x4 g, const f32x4 e, float eta, int64_t i0, int64_t d, int m,
                                                 const int js[4], const SegConst *__restrict__ crow, int s,
                                                 uint32_t k0, uint32_t k1, uint32_t t) {
    QuadCodes o;
    o.sign_nib = 0u;
    o.levels = 0u;
    u32x4 rnd;
    if (KIND == kQsgd || KIND == kMbit) {
        const uint64_t blk = static_cast<uint64_t>(i0) >> 2;
        rnd = philox4x32_10(static_cast<uint32_t>(blk), static_cast<uint32_t>(m), t, static_cast<uint32_t>(blk >> 32),
                            k0, k1);
    }
    const float fs = static_cast<float>(s);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const float gc = elem(g, c), ec = elem(e, c);
        const float egc = mul_rn(eta, gc);
        const float p = add_rn(egc, ec);
        float q = 0.0f, en = ec, egk = 0.0f;
        uint32_t neg = 0u, level = 0u;
        if (i0 + c < d) {
            egk = egc;
            neg = signbit(p) ? 1u : 0u;
            if (KIND == kSign) {
                const float sc = crow[js[c]].a;
                q = neg ? -sc : sc;
            } else if (KIND == kQsgd || KIND == kMbit) {
                const SegConst cs = crow[js[c]];
                const float a = fabsf(p);
                if (cs.a != 0.0f && a > 0.0f) {
                    const float r = level_ratio(a, cs.a);
                    const float l = fminf(floorf(r), fs);
                    const float frac = (l == fs) ? 0.0f : sub_rn(r, l);
                    const float u = static_cast<float>(elem(rnd, c) >> 8) * 0x1.0p-24f;
                    int lv = static_cast<int>(l) + ((u < frac) ? 1 : 0);
                    lv = lv > s ? s : lv;
                    level = static_cast<uint32_t>(lv);
                }
                q = copysignf(level_magnitude(level, cs.b), p);
            } else {
                q = p;
            }
            en = sub_rn(p, q);
        }
        set_elem(o.eg, c, egk);
        set_elem(o.phat, c, q);
        set_elem(o.enew, c, en);
        o.sign_nib |= neg << c;
        o.levels |= level << (8 * c);
    }
    return o;
}

// Top-k (Theorem 1): p-hat = p on the selected elements, 0 elsewhere;
// sign_nib carries the selection mask of the quad.
__device__ __forceinline__ QuadCodes encode_quad_topk(const f32x4 g, const f32x4 e, float eta, int64_t i0, int64_t d,
                                                      uint32_t T, uint32_t I) {
    QuadCodes o;
    o.sign_nib = 0u;
    o.levels = 0u;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const float gc = elem(g, c), ec = elem(e, c);
        const float egc = mul_rn(eta, gc);
        const float p = add_rn(egc, ec);
        float q = 0.0f, en = ec, egk = 0.0f;
        const int64_t i = i0 + c;
        if (i < d) {
            egk = egc;
            const uint32_t key = __float_as_uint(p) & 0x7FFFFFFFu;
            const bool sel = key > T || (key == T && static_cast<uint32_t>(i) <= I);
            q = sel ? p : 0.0f;
            en = sub_rn(p, q);
            o.sign_nib |= (sel ? 1u : 0u) << c;
        }
        set_elem(o.eg, c, egk);
        set_elem(o.phat, c, q);
        set_elem(o.enew, c, en);
    }
    return o;
}

// Ordered compaction of one row's selected elements of a 256-element tile
// (the wave's 64 quads, element 4*lane + c): the position is the tile's
// offset plus the number of selected elements before it in the tile.
__device__ __forceinline__ void store_topk(float *__restrict__ val_row, uint32_t *__restrict__ idx_row, int64_t k,
                                           uint32_t tile_base, int64_t i0, const QuadCodes &cq) {
    const uint32_t mask = cq.sign_nib;
    const int lane = threadIdx.x & 63;
    const uint64_t below = (uint64_t(1) << lane) - 1;
    uint32_t pre = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) pre += __popcll(__ballot((mask >> c) & 1u) & below);
    // Store round r writes each lane's r-th selected element: at a low
    // selection density almost every wave needs one round (two store
    // instructions) instead of one per element position of the quad.
    const uint32_t n_sel = __popc(mask);
    uint32_t rest = mask;
    for (uint32_t r = 0; __ballot(r < n_sel) != 0; ++r) {
        if (r < n_sel) {
            const int c = __ffs(rest) - 1;
            rest &= rest - 1;
            const int64_t pos = static_cast<int64_t>(tile_base) + pre + r;
            if (pos < k) {
                val_row[pos] = elem(cq.phat, c);
                idx_row[pos] = static_cast<uint32_t>(i0 + c);
            }
        }
    }
}

__device__ __forceinline__ void lookup_segments(const int64_t *__restrict__ off, const int32_t *__restrict__ tile_seg,
                                                int64_t i0, int64_t d, int js[4]) {
    const int64_t last = d - 1;
    int j = tile_seg[i0 >> 10];
    j = seg_from(off, j, i0 < last ? i0 : last);
    js[0] = j;
#pragma unroll
    for (int c = 1; c < 4; ++c) {
        const int64_t i = i0 + c;
        j = seg_from(off, j, i < last ? i : last);
        js[c] = j;
    }
}

// Message stores for one quad of one row (every lane of the wave active);
// STREAM: an 8-bit plane larger than the Infinity Cache (store_fields32).
template <int KIND, int LB, bool STREAM>
__device__ __forceinline__ void store_message(uint32_t *__restrict__ sign_row, uint32_t *__restrict__ level_row,
                                              float *__restrict__ val_row, int64_t q, const QuadCodes &cq) {
    if (KIND == kSign || KIND == kQsgd) {
        // the word of each 8-lane group (32 elements), then the four words of
        // lanes 4, 12, 20, 28 (and 36 .. 60) gathered into one 16-byte store:
        // 0.5 % faster than eight 4-byte stores (32 workers x 2^25 elements
        // and 16 x 6.3M); as a non-temporal store 3 % slower
        const uint32_t word = or_reduce8_to_lane4(cq.sign_nib << (4 * (q & 7)));
        u32x4 v4;
        v4.x = word;
        v4.y = static_cast<uint32_t>(__shfl_down(static_cast<int>(word), 8));
        v4.z = static_cast<uint32_t>(__shfl_down(static_cast<int>(word), 16));
        v4.w = static_cast<uint32_t>(__shfl_down(static_cast<int>(word), 24));
        if ((q & 31) == 4) *reinterpret_cast<u32x4 *>(sign_row + (q >> 3)) = v4;
    }
    if (KIND == kQsgd) {
        if (LB == 8) {
            store_fields32<STREAM>(level_row, q, cq.levels);
        } else {
            const uint32_t l = cq.levels;
            store_fields16(level_row, q, (l & 0xFu) | ((l >> 4) & 0xF0u) | ((l >> 8) & 0xF00u) | ((l >> 12) & 0xF000u));
        }
    }
    if (KIND == kMbit) {
        // m-bit sign-magnitude codes: the sign bit on top of each field
        const uint32_t nib = cq.sign_nib, l = cq.levels;
        if (LB == 8) {
            const uint32_t code = l | ((nib & 1u) << 7) | ((nib & 2u) << 14) | ((nib & 4u) << 21) | ((nib & 8u) << 28);
            store_fields32<STREAM>(level_row, q, code);
        } else {
            store_fields16(level_row, q,
                           (l & 0x7u) | ((l >> 4) & 0x70u) | ((l >> 8) & 0x700u) | ((l >> 12) & 0x7000u) |
                               ((nib & 1u) << 3) | ((nib & 2u) << 6) | ((nib & 4u) << 9) | ((nib & 8u) << 12));
        }
    }
    if (KIND == kIdentity) st4(val_row + 4 * q, cq.phat);
}

// store_message with the store kind chosen at run time (kernels off the
// fused step's hot loop).
template <int KIND, int LB>
__device__ __forceinline__ void store_message_rt(uint32_t *__restrict__ sign_row, uint32_t *__restrict__ level_row,
                                                 float *__restrict__ val_row, int64_t q, const QuadCodes &cq,
                                                 bool stream) {
    if (stream)
        store_message<KIND, LB, true>(sign_row, level_row, val_row, q, cq);
    else
        store_message<KIND, LB, false>(sign_row, level_row, val_row, q, cq);
}

struct RowArgs {
    float eta;
    uint32_t t;
    int64_t d, ld;
    int32_t M, n_seg, s;
    uint32_t k0, k1;
    int64_t sign_words, level_words;  // words per row of each plane
    int32_t stream_msg;               // message planes larger than the Infinity Cache: streaming stores
};

// Worker side only (dqgan_compress_ef): one quad per thread for kEncRows
// consecutive workers, whose g and e are all loaded before the first is
// encoded (more loads in flight per lane).
constexpr int kEncRows = 4;

template <int KIND, int LB>
__global__ __launch_bounds__(kBlock) void k_encode_rows(const float *__restrict__ G, float *__restrict__ E,
                                                        uint32_t *__restrict__ sign_plane,
                                                        uint32_t *__restrict__ level_plane, float *__restrict__ val,
                                                        const SegConst *__restrict__ consts,
                                                        const int64_t *__restrict__ off,
                                                        const int32_t *__restrict__ tile_seg, RowArgs a) {
    const int64_t q = static_cast<int64_t>(blockIdx.x) * kQuadsPerBlock + threadIdx.x;
    const int m0 = static_cast<int>(blockIdx.y) * kEncRows;
    const int64_t i0 = 4 * q;
    int js[4];
    lookup_segments(off, tile_seg, i0, a.d, js);
    const int j_first = __builtin_amdgcn_readfirstlane(js[0]);
    const bool one_seg = __ballot(js[0] != j_first || js[3] != j_first) == 0;
    const int z[4] = {0, 0, 0, 0};
    f32x4 gv[kEncRows], ev[kEncRows];
#pragma unroll
    for (int u = 0; u < kEncRows; ++u) {
        const int m = m0 + u;
        if (m < a.M) {
            const int64_t rb = static_cast<int64_t>(m) * a.ld;
            gv[u] = ld_stream(G + rb + i0);
            ev[u] = ld_stream(E + rb + i0);
        }
    }
#pragma unroll
    for (int u = 0; u < kEncRows; ++u) {
        const int m = m0 + u;
        if (m < a.M) {
            const int64_t rb = static_cast<int64_t>(m) * a.ld;
            const SegConst *crow = consts + static_cast<int64_t>(m) * a.n_seg;
            QuadCodes cq;
            if (one_seg) {
                const SegConst c1[1] = {crow[j_first]};
                cq = encode_quad<KIND>(gv[u], ev[u], a.eta, i0, a.d, m, z, c1, a.s, a.k0, a.k1, a.t);
            } else {
                cq = encode_quad<KIND>(gv[u], ev[u], a.eta, i0, a.d, m, js, crow, a.s, a.k0, a.k1, a.t);
            }
            st_stream(E + rb + i0, cq.enew);
            store_message_rt<KIND, LB>(sign_plane + m * a.sign_words, level_plane + m * a.level_words, val + rb, q,
                                       cq, a.stream_msg != 0);
        }
    }
}

// The fused step.  MT > 0: M == MT, the extrapolation operands stay in
// registers; MT == 0: any M, the second sweep re-reads g and the new e.
template <int KIND, int LB, int MT>
__global__ __launch_bounds__(kBlock) void k_fused(const float *__restrict__ G, float *__restrict__ E,
                                                  float *__restrict__ W, float *__restrict__ WX,
                                                  float *__restrict__ Qhat, uint32_t *__restrict__ sign_plane,
                                                  uint32_t *__restrict__ level_plane, float *__restrict__ val,
                                                  const SegConst *__restrict__ consts, const int64_t *__restrict__ off,
                                                  const int32_t *__restrict__ tile_seg, RowArgs a, float invM,
                                                  TopkArgs ta) {
    const int64_t q = static_cast<int64_t>(blockIdx.x) * kQuadsPerBlock + threadIdx.x;
    const int64_t i0 = 4 * q;
    // top-k: each wave's 64 quads are one counting tile
    const int64_t tile = static_cast<int64_t>(blockIdx.x) * (kQuadsPerBlock / 64) + (threadIdx.x >> 6);
    const int M = MT > 0 ? MT : a.M;
    constexpr int kUnroll = MT > 0 ? MT : 1;
    int js[4];
    lookup_segments(off, tile_seg, i0, a.d, js);
    f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
    f32x4 xs[MT > 0 ? MT : 1];
#pragma unroll kUnroll
    for (int m = 0; m < M; ++m) {
        const int64_t rb = static_cast<int64_t>(m) * a.ld;
        const f32x4 g = ld_stream(G + rb + i0);
        const f32x4 e = ld_stream(E + rb + i0);
        QuadCodes cq;
        if constexpr (KIND == kTopk) {
            const TopkRow *rw = ta.rows + m;
            cq = encode_quad_topk(g, e, a.eta, i0, a.d, rw->T, rw->I);
        } else {
            cq = encode_quad<KIND>(g, e, a.eta, i0, a.d, m, js, consts + static_cast<int64_t>(m) * a.n_seg, a.s, a.k0,
                                   a.k1, a.t);
        }
        st_stream(E + rb + i0, cq.enew);
        if constexpr (KIND == kTopk) {
            store_topk(val + m * ta.k, ta.idx + m * ta.k, ta.k, topk_tile_base(ta, m, tile), i0, cq);
        } else {
            store_message_rt<KIND, LB>(sign_plane + m * a.sign_words, level_plane + m * a.level_words, val + rb, q, cq,
                                       a.stream_msg != 0);
        }
        if (m == 0) {
            acc = cq.phat;
        } else {
#pragma unroll
            for (int c = 0; c < 4; ++c) set_elem(acc, c, add_rn(elem(acc, c), elem(cq.phat, c)));
        }
        if (MT > 0) {
            f32x4 x;
#pragma unroll
            for (int c = 0; c < 4; ++c) set_elem(x, c, add_rn(elem(cq.eg, c), elem(cq.enew, c)));
            xs[MT > 0 ? m : 0] = x;
        }
    }
    f32x4 qh;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const float sacc = elem(acc, c);
        const float v = invM > 0.0f ? mul_rn(sacc, invM)
                                    : static_cast<float>(static_cast<double>(sacc) / static_cast<double>(M));
        set_elem(qh, c, v);
    }
    const f32x4 w = ld4(W + i0);
    f32x4 wt;
#pragma unroll
    for (int c = 0; c < 4; ++c) set_elem(wt, c, sub_rn(elem(w, c), elem(qh, c)));
    st4(W + i0, wt);
    if (Qhat) st4(Qhat + i0, qh);
#pragma unroll kUnroll
    for (int m = 0; m < M; ++m) {
        const int64_t rb = static_cast<int64_t>(m) * a.ld;
        f32x4 x;
        if (MT > 0) {
            x = xs[MT > 0 ? m : 0];
        } else {
            const f32x4 g = ld4(G + rb + i0);
            const f32x4 en = ld4(E + rb + i0);
#pragma unroll
            for (int c = 0; c < 4; ++c) set_elem(x, c, add_rn(mul_rn(a.eta, elem(g, c)), elem(en, c)));
        }
        f32x4 wx;
#pragma unroll
        for (int c = 0; c < 4; ++c) set_elem(wx, c, (i0 + c < a.d) ? sub_rn(elem(wt, c), elem(x, c)) : 0.0f);
        st_stream(WX + rb + i0, wx);
    }
}

// The fused step with the rows split across the NG waves of a workgroup:
// all waves cover the same 64 quads, wave g owns rows g*R .. g*R+R-1 (rows
// at or beyond M are skipped) and keeps only their p-hat and extrapolation
// operands in registers.  The server sum runs in ascending worker order as a
// chain through LDS: wave g adds its rows to the partial sum of waves
// 0..g-1, so the result is the same sequential binary32 sum as in the
// one-lane-per-quad kernel.  Few registers per lane leave room for many
// waves per SIMD, which keeps enough loads in flight to stream from HBM.
template <int KIND, int LB, int R, int NG, bool STREAM>
__global__ __launch_bounds__(64 * NG) void k_fused_split(const float *__restrict__ G, float *__restrict__ E,
                                                         float *__restrict__ W, float *__restrict__ WX,
                                                         float *__restrict__ Qhat, uint32_t *__restrict__ sign_plane,
                                                         uint32_t *__restrict__ level_plane, float *__restrict__ val,
                                                         const SegConst *__restrict__ consts,
                                                         const int64_t *__restrict__ off,
                                                         const int32_t *__restrict__ tile_seg, RowArgs a, float invM,
                                                         TopkArgs ta) {
    __shared__ f32x4 chain[64];
    const int lane = threadIdx.x & 63;
    const int g = __builtin_amdgcn_readfirstlane(static_cast<int>(threadIdx.x >> 6));
    const int M = a.M;
    const int last_g = (M - 1) / R;  // the wave that finishes the sum
    const int64_t q = static_cast<int64_t>(blockIdx.x) * 64 + lane;
    const int64_t i0 = 4 * q;
    int js[4];
    lookup_segments(off, tile_seg, i0, a.d, js);
    // One segment for the whole wave (the common case): its constants are
    // fetched with one scalar load per row.
    const int j_first = __builtin_amdgcn_readfirstlane(js[0]);
    const bool one_seg = __ballot(js[0] != j_first || js[3] != j_first) == 0;
    f32x4 ph[R], xs[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int m = g * R + r;
        if (m < M) {
            const int64_t rb = static_cast<int64_t>(m) * a.ld;
            const f32x4 gv = ld_stream(G + rb + i0);
            const f32x4 ev = ld_stream(E + rb + i0);
            const SegConst *crow = consts + static_cast<int64_t>(m) * a.n_seg;
            QuadCodes cq;
            if constexpr (KIND == kTopk) {
                const TopkRow *rw = ta.rows + m;
                cq = encode_quad_topk(gv, ev, a.eta, i0, a.d, rw->T, rw->I);
            } else if (one_seg) {
                const SegConst cu = crow[j_first];
                const SegConst c4[1] = {cu};
                const int z[4] = {0, 0, 0, 0};
                cq = encode_quad<KIND>(gv, ev, a.eta, i0, a.d, m, z, c4, a.s, a.k0, a.k1, a.t);
            } else {
                cq = encode_quad<KIND>(gv, ev, a.eta, i0, a.d, m, js, crow, a.s, a.k0, a.k1, a.t);
            }
            st_stream(E + rb + i0, cq.enew);
            if constexpr (KIND == kTopk) {
                store_topk(val + m * ta.k, ta.idx + m * ta.k, ta.k, topk_tile_base(ta, m, blockIdx.x), i0, cq);
            } else {
                store_message<KIND, LB, STREAM>(sign_plane + m * a.sign_words, level_plane + m * a.level_words,
                                                val + rb, q, cq);
            }
            ph[r] = cq.phat;
#pragma unroll
            for (int c = 0; c < 4; ++c) set_elem(xs[r], c, add_rn(elem(cq.eg, c), elem(cq.enew, c)));
        }
    }
#pragma unroll
    for (int phase = 0; phase < NG; ++phase) {
        if (phase <= last_g) {
            if (g == phase) {
                f32x4 acc;
                if (phase == 0) {
                    acc = ph[0];
                } else {
                    acc = chain[lane];
#pragma unroll
                    for (int c = 0; c < 4; ++c) set_elem(acc, c, add_rn(elem(acc, c), elem(ph[0], c)));
                }
#pragma unroll
                for (int r = 1; r < R; ++r) {
                    if (g * R + r < M) {
#pragma unroll
                        for (int c = 0; c < 4; ++c) set_elem(acc, c, add_rn(elem(acc, c), elem(ph[r], c)));
                    }
                }
                if (phase < last_g) {
                    chain[lane] = acc;
                } else {
                    f32x4 qh;
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        const float sacc = elem(acc, c);
                        set_elem(qh, c, invM > 0.0f ? mul_rn(sacc, invM)
                                                    : static_cast<float>(static_cast<double>(sacc) /
                                                                         static_cast<double>(M)));
                    }
                    const f32x4 w = ld4(W + i0);
                    f32x4 wt;
#pragma unroll
                    for (int c = 0; c < 4; ++c) set_elem(wt, c, sub_rn(elem(w, c), elem(qh, c)));
                    st4(W + i0, wt);
                    if (Qhat) st4(Qhat + i0, qh);
                    chain[lane] = wt;
                }
            }
            __syncthreads();
        }
    }
    const f32x4 wt = chain[lane];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int m = g * R + r;
        if (m < M) {
            const int64_t rb = static_cast<int64_t>(m) * a.ld;
            f32x4 wx;
#pragma unroll
            for (int c = 0; c < 4; ++c) set_elem(wx, c, (i0 + c < a.d) ? sub_rn(elem(wt, c), elem(xs[r], c)) : 0.0f);
            st_stream(WX + rb + i0, wx);
        }
    }
}

// Decode one quad of one row's message to p-hat from its fields: nib = the
// four sign bits (SIGN, QSGD), raw = the quad's level or code bits (QSGD,
// MBIT: 32 bits for 8-bit fields, the low 16 for 4-bit fields).
// CHECK_D: elements at or beyond d decode to 0 (only the last quads of a
// row need it).  The magnitude is never negative, so the sign bit is set by
// OR (-0 for a zero level with the sign bit set, as the encoder gives).
template <int KIND, int LB, bool CHECK_D = true>
__device__ __forceinline__ f32x4 decode_fields(uint32_t nib, uint32_t raw, const SegConst *__restrict__ crow,
                                               const int js[4], int64_t i0, int64_t d) {
    f32x4 out = {0.0f, 0.0f, 0.0f, 0.0f};
    uint32_t lev = 0u;
    if (KIND == kMbit) {
        if (LB == 8) {
            lev = raw & 0x7F7F7F7Fu;
            nib = ((raw >> 7) & 1u) | ((raw >> 14) & 2u) | ((raw >> 21) & 4u) | ((raw >> 28) & 8u);
        } else {
            lev = (raw & 0x7u) | ((raw & 0x70u) << 4) | ((raw & 0x700u) << 8) | ((raw & 0x7000u) << 12);
            nib = ((raw >> 3) & 1u) | ((raw >> 6) & 2u) | ((raw >> 9) & 4u) | ((raw >> 12) & 8u);
        }
    }
    if (KIND == kQsgd) {
        if (LB == 8)
            lev = raw;
        else
            lev = (raw & 0xFu) | ((raw & 0xF0u) << 4) | ((raw & 0xF00u) << 8) | ((raw & 0xF000u) << 12);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        if (CHECK_D && i0 + c >= d) continue;
        float mag;
        if (KIND == kSign) {
            mag = crow[js[c]].a;
        } else {
            const uint32_t l = (lev >> (8 * c)) & 0xFFu;
            mag = level_magnitude(l, crow[js[c]].b);
        }
        set_elem(out, c, __uint_as_float(__float_as_uint(mag) | (((nib >> c) & 1u) << 31)));
    }
    return out;
}

// Decode one quad of one row's message to p-hat.
template <int KIND, int LB>
__device__ __forceinline__ f32x4 decode_quad(const uint32_t *__restrict__ sign_row, const uint32_t *__restrict__ level_row,
                                             const float *__restrict__ val_row, const SegConst *__restrict__ crow,
                                             int64_t q, int64_t d, const int js[4]) {
    const int64_t i0 = 4 * q;
    if (KIND == kIdentity) {
        const f32x4 v = ld4(val_row + i0);
        f32x4 out;
#pragma unroll
        for (int c = 0; c < 4; ++c) set_elem(out, c, (i0 + c < d) ? elem(v, c) : 0.0f);
        return out;
    }
    const uint32_t nib = (KIND == kSign || KIND == kQsgd) ? (sign_row[q >> 3] >> (4 * (q & 7))) & 0xFu : 0u;
    uint32_t raw = 0u;
    if (KIND == kQsgd || KIND == kMbit)
        raw = LB == 8 ? level_row[q] : static_cast<uint32_t>(reinterpret_cast<const uint16_t *>(level_row)[q]);
    return decode_fields<KIND, LB>(nib, raw, crow, js, i0, d);
}

template <int KIND, int LB>
__global__ __launch_bounds__(kBlock) void k_unpack(const uint32_t *__restrict__ sign_plane,
                                                   const uint32_t *__restrict__ level_plane,
                                                   const float *__restrict__ val, float *__restrict__ Phat,
                                                   const SegConst *__restrict__ consts, const int64_t *__restrict__ off,
                                                   const int32_t *__restrict__ tile_seg, RowArgs a) {
    const int64_t q = static_cast<int64_t>(blockIdx.x) * kQuadsPerBlock + threadIdx.x;
    const int m = blockIdx.y;
    const int64_t rb = static_cast<int64_t>(m) * a.ld;
    int js[4];
    lookup_segments(off, tile_seg, 4 * q, a.d, js);
    const f32x4 v = decode_quad<KIND, LB>(sign_plane + m * a.sign_words, level_plane + m * a.level_words, val + rb,
                                          consts + static_cast<int64_t>(m) * a.n_seg, q, a.d, js);
    st_stream(Phat + rb + 4 * q, v);
}

// Server average of the M messages.  A thread covers four consecutive
// quads (16 elements: 16 sign bits, 8 or 16 bytes of fields per row, so
// each row's loads are 2-16 bytes per lane rather than sub-word), and takes
// the rows in chunks of kAggRows whose fields are all loaded before the
// first is decoded; the sum runs in ascending worker order.
constexpr int kAggQuads = 4;
constexpr int kAggRows = 4;

template <int KIND, int LB>
__global__ __launch_bounds__(kBlock) void k_aggregate(const uint32_t *__restrict__ sign_plane,
                                                      const uint32_t *__restrict__ level_plane,
                                                      const float *__restrict__ val, float *__restrict__ Qhat,
                                                      const SegConst *__restrict__ consts,
                                                      const int64_t *__restrict__ off,
                                                      const int32_t *__restrict__ tile_seg, RowArgs a, float invM) {
    const int64_t g16 = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;  // group of 16 elements
    const int64_t q0 = kAggQuads * g16;
    const bool live = 4 * q0 < a.ld;
    int js[kAggQuads][4];
#pragma unroll
    for (int k = 0; k < kAggQuads; ++k) lookup_segments(off, tile_seg, live ? 4 * (q0 + k) : 0, a.d, js[k]);
    // the whole wave in one segment (the common case): one scalar load of
    // the constants per row
    const int j_first = __builtin_amdgcn_readfirstlane(js[0][0]);
    const bool one_seg = __ballot(live && (js[0][0] != j_first || js[kAggQuads - 1][3] != j_first)) == 0;
    const int z[4] = {0, 0, 0, 0};
    // every element of the wave below d: no per-element bound tests
    const bool full = __ballot(4 * (q0 + kAggQuads) > a.d) == 0;
    constexpr int kFieldWords = (KIND == kQsgd || KIND == kMbit) ? LB / 2 : 0;  // 32-bit words of fields per row
    f32x4 acc[kAggQuads];
#pragma unroll
    for (int k = 0; k < kAggQuads; ++k) acc[k] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    // the fields of row m for this thread's 16 elements
    auto load_row = [&](int m, uint32_t &sg, uint32_t (&fw)[kFieldWords > 0 ? kFieldWords : 1],
                        f32x4 (&vv)[KIND == kIdentity ? kAggQuads : 1]) {
        if (KIND == kSign || KIND == kQsgd) sg = reinterpret_cast<const uint16_t *>(sign_plane + m * a.sign_words)[g16];
        if (kFieldWords == 4) {
            const u32x4 v = *reinterpret_cast<const u32x4 *>(level_plane + m * a.level_words + 4 * g16);
            fw[0] = v.x;
            fw[kFieldWords > 1 ? 1 : 0] = v.y;
            fw[kFieldWords > 2 ? 2 : 0] = v.z;
            fw[kFieldWords > 3 ? 3 : 0] = v.w;
        } else if (kFieldWords == 2) {
            const uint2 v = *reinterpret_cast<const uint2 *>(level_plane + m * a.level_words + 2 * g16);
            fw[0] = v.x;
            fw[kFieldWords > 1 ? 1 : 0] = v.y;
        }
        if (KIND == kIdentity) {
#pragma unroll
            for (int k = 0; k < kAggQuads; ++k)
                vv[KIND == kIdentity ? k : 0] = ld4(val + static_cast<int64_t>(m) * a.ld + 4 * (q0 + k));
        }
    };
    // add row m (ascending order) given its loaded fields and its constants
    auto add_row = [&](int m, uint32_t sg, const uint32_t (&fw)[kFieldWords > 0 ? kFieldWords : 1],
                       const f32x4 (&vv)[KIND == kIdentity ? kAggQuads : 1], const SegConst *crow, bool uniform) {
#pragma unroll
        for (int k = 0; k < kAggQuads; ++k) {
            const int64_t i0 = 4 * (q0 + k);
            f32x4 v;
            if (KIND == kIdentity) {
#pragma unroll
                for (int c = 0; c < 4; ++c) set_elem(v, c, (i0 + c < a.d) ? elem(vv[KIND == kIdentity ? k : 0], c) : 0.0f);
            } else {
                const uint32_t nib = (KIND == kSign || KIND == kQsgd) ? (sg >> (4 * k)) & 0xFu : 0u;
                uint32_t raw = 0u;
                if (kFieldWords == 4) raw = fw[k < kFieldWords ? k : 0];
                if (kFieldWords == 2) raw = (fw[(k >> 1) < kFieldWords ? (k >> 1) : 0] >> (16 * (k & 1))) & 0xFFFFu;
                v = full ? decode_fields<KIND, LB, false>(nib, raw, crow, uniform ? z : js[k], i0, a.d)
                         : decode_fields<KIND, LB, true>(nib, raw, crow, uniform ? z : js[k], i0, a.d);
            }
            if (m == 0) {
                acc[k] = v;
            } else {
#pragma unroll
                for (int c = 0; c < 4; ++c) set_elem(acc[k], c, add_rn(elem(acc[k], c), elem(v, c)));
            }
        }
    };
    if (one_seg) {
        // kAggRows rows' fields loaded before the first is decoded
        for (int m0 = 0; m0 < a.M; m0 += kAggRows) {
            uint32_t sg[kAggRows];
            uint32_t fw[kAggRows][kFieldWords > 0 ? kFieldWords : 1];
            f32x4 vv[kAggRows][KIND == kIdentity ? kAggQuads : 1];
#pragma unroll
            for (int u = 0; u < kAggRows; ++u)
                if (m0 + u < a.M && live) load_row(m0 + u, sg[u], fw[u], vv[u]);
#pragma unroll
            for (int u = 0; u < kAggRows; ++u) {
                const int m = m0 + u;
                if (m < a.M && live) {
                    const SegConst c1[1] = {consts[static_cast<int64_t>(m) * a.n_seg + j_first]};
                    add_row(m, sg[u], fw[u], vv[u], c1, true);
                }
            }
        }
    } else if (live) {
        // a wave across segment boundaries: one row at a time
        for (int m = 0; m < a.M; ++m) {
            uint32_t sg = 0u;
            uint32_t fw[kFieldWords > 0 ? kFieldWords : 1];
            f32x4 vv[KIND == kIdentity ? kAggQuads : 1];
            load_row(m, sg, fw, vv);
            add_row(m, sg, fw, vv, consts + static_cast<int64_t>(m) * a.n_seg, false);
        }
    }
    if (!live) return;
#pragma unroll
    for (int k = 0; k < kAggQuads; ++k) {
        f32x4 qh;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float sacc = elem(acc[k], c);
            set_elem(qh, c, invM > 0.0f ? mul_rn(sacc, invM)
                                        : static_cast<float>(static_cast<double>(sacc) / static_cast<double>(a.M)));
        }
        st4(Qhat + 4 * (q0 + k), qh);
    }
}

__global__ __launch_bounds__(kBlock) void k_omd(const float *__restrict__ Qhat, float *__restrict__ W,
                                                const float *__restrict__ G, const float *__restrict__ E,
                                                float *__restrict__ WX, float eta, int64_t d, int64_t ld, int32_t M) {
    const int64_t q = static_cast<int64_t>(blockIdx.x) * kQuadsPerBlock + threadIdx.x;
    const int64_t i0 = 4 * q;
    const f32x4 w = ld4(W + i0);
    const f32x4 qh = ld4(Qhat + i0);
    f32x4 wt;
#pragma unroll
    for (int c = 0; c < 4; ++c) set_elem(wt, c, (i0 + c < d) ? sub_rn(elem(w, c), elem(qh, c)) : elem(w, c));
    st4(W + i0, wt);
    if (!WX) return;
    // kOmdRows workers' g and e loaded before the first evaluation point
    constexpr int kOmdRows = 4;
    for (int m0 = 0; m0 < M; m0 += kOmdRows) {
        f32x4 gv[kOmdRows], ev[kOmdRows];
#pragma unroll
        for (int u = 0; u < kOmdRows; ++u) {
            if (m0 + u < M) {
                const int64_t rb = static_cast<int64_t>(m0 + u) * ld;
                gv[u] = ld_stream(G + rb + i0);
                ev[u] = ld_stream(E + rb + i0);
            }
        }
#pragma unroll
        for (int u = 0; u < kOmdRows; ++u) {
            if (m0 + u < M) {
                f32x4 wx;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const float x = add_rn(mul_rn(eta, elem(gv[u], c)), elem(ev[u], c));
                    set_elem(wx, c, (i0 + c < d) ? sub_rn(elem(wt, c), x) : 0.0f);
                }
                st_stream(WX + static_cast<int64_t>(m0 + u) * ld + i0, wx);
            }
        }
    }
}

template <int LB, int KIND>
__global__ __launch_bounds__(kBlock) void k_pack(const uint16_t *__restrict__ codes, uint32_t *__restrict__ sign_plane,
                                                 uint32_t *__restrict__ level_plane, RowArgs a) {
    const int64_t q = static_cast<int64_t>(blockIdx.x) * kQuadsPerBlock + threadIdx.x;
    const int m = blockIdx.y;
    const int64_t i0 = 4 * q;
    const uint2 raw = *reinterpret_cast<const uint2 *>(codes + static_cast<int64_t>(m) * a.ld + i0);
    const uint32_t c4[4] = {raw.x & 0xFFFFu, raw.x >> 16, raw.y & 0xFFFFu, raw.y >> 16};
    QuadCodes cq;
    cq.sign_nib = 0u;
    cq.levels = 0u;
    const uint32_t fmask = KIND == kMbit ? (LB == 8 ? 0x7Fu : 0x7u) : (LB == 8 ? 0xFFu : 0xFu);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        if (i0 + c >= a.d) continue;
        cq.sign_nib |= ((c4[c] >> 15) & 1u) << c;
        cq.levels |= (c4[c] & fmask) << (8 * c);
    }
    if (KIND == kSign)
        store_message_rt<kSign, 0>(sign_plane + m * a.sign_words, nullptr, nullptr, q, cq, a.stream_msg != 0);
    else if (KIND == kMbit)
        store_message_rt<kMbit, LB>(nullptr, level_plane + m * a.level_words, nullptr, q, cq, a.stream_msg != 0);
    else
        store_message_rt<kQsgd, LB>(sign_plane + m * a.sign_words, level_plane + m * a.level_words, nullptr, q,
                                    cq, a.stream_msg != 0);
}

// Top-k worker side only (dqgan_compress_ef): one wave per (tile, worker).
__global__ __launch_bounds__(64) void k_topk_encode_rows(const float *__restrict__ G, float *__restrict__ E,
                                                         float *__restrict__ val, RowArgs a, TopkArgs ta) {
    const int m = blockIdx.y;
    const int64_t q = static_cast<int64_t>(blockIdx.x) * 64 + threadIdx.x;
    const int64_t i0 = 4 * q;
    const int64_t rb = static_cast<int64_t>(m) * a.ld;
    const TopkRow *rw = ta.rows + m;
    const f32x4 g = ld_stream(G + rb + i0);
    const f32x4 e = ld_stream(E + rb + i0);
    const QuadCodes cq = encode_quad_topk(g, e, a.eta, i0, a.d, rw->T, rw->I);
    st_stream(E + rb + i0, cq.enew);
    store_topk(val + m * ta.k, ta.idx + m * ta.k, ta.k, topk_tile_base(ta, m, blockIdx.x), i0, cq);
}

RowArgs row_args(const dqgan_plan_s &P, float eta, uint32_t t) {
    RowArgs a;
    a.eta = eta;
    a.t = t;
    a.d = P.desc.d;
    a.ld = P.desc.ld;
    a.M = P.desc.M;
    a.n_seg = P.desc.n_seg;
    a.s = P.level_count;
    a.k0 = static_cast<uint32_t>(P.desc.seed);
    a.k1 = static_cast<uint32_t>(P.desc.seed >> 32);
    a.sign_words = P.desc.ld / 32;
    a.level_words = P.level_bits ? P.desc.ld * P.level_bits / 32 : 0;
    const double msg_bytes = 4.0 * P.desc.M * static_cast<double>(a.sign_words + a.level_words);
    a.stream_msg = msg_bytes > kInfinityCacheBytes ? 1 : 0;
    return a;
}

// 1/M when M is a power of two (then x * (1/M) equals x / M exactly),
// else 0 (the kernels divide).
float inv_m(int M) { return (M & (M - 1)) == 0 ? 1.0f / static_cast<float>(M) : 0.0f; }

// The state the top-k apply pass reads (threshold per row, tile offsets).
TopkArgs topk_args(const dqgan_plan_s &P, const dqgan_wire &w) {
    TopkArgs ta{};
    if (P.desc.kind == kTopk) {
        ta.rows = P.topk.rows;
        ta.tile_off = P.topk.tile_off;
        ta.chunk_off = P.topk.chunk_off;
        ta.n_tiles = P.topk.n_tiles;
        ta.n_chunks = P.topk.n_chunks;
        ta.k = P.desc.k;
        ta.idx = w.idx;
    }
    return ta;
}

template <int KIND, int LB, int MT>
hipError_t fused_launch(const dqgan_plan_s &P, const RowArgs &a, const float *G, float *E, float *W, float *WX,
                        const dqgan_wire &w, float *Qhat, hipStream_t st) {
    hipLaunchKernelGGL((k_fused<KIND, LB, MT>), dim3(static_cast<unsigned>(P.n_tiles)), dim3(kBlock), 0, st, G, E, W,
                       WX, Qhat, w.sign, w.level, w.val, P.d_consts, P.d_off, P.d_tile_seg, a, inv_m(P.desc.M),
                       topk_args(P, w));
    return hipGetLastError();
}

template <int KIND, int LB, int R, int NG>
hipError_t split_launch(const dqgan_plan_s &P, const RowArgs &a, const float *G, float *E, float *W, float *WX,
                        const dqgan_wire &w, float *Qhat, hipStream_t st) {
    if (P.desc.M > R * NG) return hipErrorInvalidValue;  // every worker must belong to a wave
    const TopkArgs ta = topk_args(P, w);
    const dim3 grid(static_cast<unsigned>(P.n_tiles * 4)), block(64 * NG);
    // Only 8-bit planes have a second store kind (store_fields32).
    constexpr bool kTwoKinds = (KIND == kQsgd || KIND == kMbit) && LB == 8;
    if (kTwoKinds && a.stream_msg)
        hipLaunchKernelGGL((k_fused_split<KIND, LB, R, NG, kTwoKinds>), grid, block, 0, st, G, E, W, WX, Qhat, w.sign,
                           w.level, w.val, P.d_consts, P.d_off, P.d_tile_seg, a, inv_m(P.desc.M), ta);
    else
        hipLaunchKernelGGL((k_fused_split<KIND, LB, R, NG, false>), grid, block, 0, st, G, E, W, WX, Qhat, w.sign,
                           w.level, w.val, P.d_consts, P.d_off, P.d_tile_seg, a, inv_m(P.desc.M), ta);
    return hipGetLastError();
}

// Launch shape of the fused step: up to 16 waves per workgroup, each owning
// R rows; more rows per wave means more loads in flight per lane.  Measured:
// for 9 <= M <= 16, 8 waves x 2 rows beats 16 x 1 by 10-13 %; for
// 17 <= M <= 32, 8 waves x 4 rows beats 16 x 2 by 2-3 % although it runs 6
// rather than 8 waves per SIMD; M <= 8 (cache-resident sizes) keeps one row
// per wave; for 65 <= M <= 128, 16 waves x 8 rows (4 waves per SIMD) is a
// third faster than the one-lane kernel.  Beyond 128 rows no register-resident
// split fits (16 rows per lane need more than the 128 VGPRs a 16-wave
// workgroup allows), and the one-lane-per-quad kernel serves.
template <int KIND, int LB>
hipError_t fused_by_m(const dqgan_plan_s &P, const RowArgs &a, const float *G, float *E, float *W, float *WX,
                      const dqgan_wire &w, float *Qhat, hipStream_t st) {
    const int M = P.desc.M;
    if (M <= 4) return split_launch<KIND, LB, 1, 4>(P, a, G, E, W, WX, w, Qhat, st);
    if (M <= 8) return split_launch<KIND, LB, 1, 8>(P, a, G, E, W, WX, w, Qhat, st);
    if (M <= 16) return split_launch<KIND, LB, 2, 8>(P, a, G, E, W, WX, w, Qhat, st);
    if (M <= 32) return split_launch<KIND, LB, 4, 8>(P, a, G, E, W, WX, w, Qhat, st);
    if (M <= 64) return split_launch<KIND, LB, 4, 16>(P, a, G, E, W, WX, w, Qhat, st);
    if (M <= 128) return split_launch<KIND, LB, 8, 16>(P, a, G, E, W, WX, w, Qhat, st);
    return fused_launch<KIND, LB, 0>(P, a, G, E, W, WX, w, Qhat, st);
}

}  // namespace

hipError_t launch_segment_scales(const dqgan_plan_s &P, float eta, const float *G, const float *E,
                                 const float *scales_in, float *scale_out, hipStream_t st) {
    const dqgan_desc &D = P.desc;
    if (!scales_in) {
        const dim3 grid(static_cast<unsigned>(P.n_pieces), static_cast<unsigned>(D.M));
        if (D.norm == DQGAN_L1)
            hipLaunchKernelGGL(k_segment_partials<DQGAN_L1>, grid, dim3(kBlock), 0, st, G, E, eta, D.ld, P.d_pieces,
                               P.n_pieces, P.d_partial, P.d_pmax);
        else if (D.norm == DQGAN_L2)
            hipLaunchKernelGGL(k_segment_partials<DQGAN_L2>, grid, dim3(kBlock), 0, st, G, E, eta, D.ld, P.d_pieces,
                               P.n_pieces, P.d_partial, P.d_pmax);
        else
            hipLaunchKernelGGL(k_segment_partials<DQGAN_LINF>, grid, dim3(kBlock), 0, st, G, E, eta, D.ld,
                               P.d_pieces, P.n_pieces, P.d_partial, P.d_pmax);
        hipError_t err = hipGetLastError();
        if (err != hipSuccess) return err;
    }
    const int64_t n = static_cast<int64_t>(D.M) * D.n_seg;
    // one wave per (worker, segment)
    hipLaunchKernelGGL(k_finalize, dim3(static_cast<unsigned>((n * 64 + kBlock - 1) / kBlock)), dim3(kBlock), 0, st, D.kind,
                       D.norm, P.level_count, P.d_partial, P.d_pmax, P.n_pieces, P.d_seg_piece, P.d_off, D.M, D.n_seg,
                       scales_in, scale_out, P.d_consts);
    return hipGetLastError();
}

hipError_t launch_consts_from_scales(const dqgan_plan_s &P, const float *scales, hipStream_t st) {
    return launch_segment_scales(P, 0.0f, nullptr, nullptr, scales, nullptr, st);
}

namespace {

// Calls f(kind, field bits) with both as compile-time constants, for the
// dense compressors: (SIGN, 0), (QSGD, 8 or 4), (MBIT, 8 or 4), (IDENTITY, 0).
template <int V>
using Const = std::integral_constant<int, V>;

template <typename F>
hipError_t with_dense_kind(const dqgan_plan_s &P, F &&f) {
    switch (P.desc.kind) {
        case kSign: return f(Const<kSign>{}, Const<0>{});
        case kQsgd: return P.level_bits == 8 ? f(Const<kQsgd>{}, Const<8>{}) : f(Const<kQsgd>{}, Const<4>{});
        case kMbit: return P.level_bits == 8 ? f(Const<kMbit>{}, Const<8>{}) : f(Const<kMbit>{}, Const<4>{});
        default: return f(Const<kIdentity>{}, Const<0>{});
    }
}

}  // namespace

hipError_t launch_encode(const dqgan_plan_s &P, float eta, uint32_t t, const float *G, float *E, const dqgan_wire &w,
                         hipStream_t st) {
    const RowArgs a = row_args(P, eta, t);
    const dim3 grid(static_cast<unsigned>(P.n_tiles), static_cast<unsigned>((P.desc.M + kEncRows - 1) / kEncRows));
    return with_dense_kind(P, [&](auto K, auto L) {
        hipLaunchKernelGGL((k_encode_rows<decltype(K)::value, decltype(L)::value>), grid, dim3(kBlock), 0, st, G, E,
                           w.sign, w.level, w.val, P.d_consts, P.d_off, P.d_tile_seg, a);
        return hipGetLastError();
    });
}

hipError_t launch_fused_dense(const dqgan_plan_s &P, float eta, uint32_t t, const float *G, float *E, float *W,
                              float *WX, const dqgan_wire &w, float *Qhat, hipStream_t st) {
    const RowArgs a = row_args(P, eta, t);
    return with_dense_kind(P, [&](auto K, auto L) {
        return fused_by_m<decltype(K)::value, decltype(L)::value>(P, a, G, E, W, WX, w, Qhat, st);
    });
}

hipError_t launch_pack(const dqgan_plan_s &P, const uint16_t *codes, const dqgan_wire &w, hipStream_t st) {
    const RowArgs a = row_args(P, 0.0f, 0);
    const dim3 grid(static_cast<unsigned>(P.n_tiles), static_cast<unsigned>(P.desc.M));
    return with_dense_kind(P, [&](auto K, auto L) {
        if constexpr (decltype(K)::value == kIdentity) {
            return hipErrorInvalidValue;  // the identity has no codes to pack
        } else {
            hipLaunchKernelGGL((k_pack<decltype(L)::value, decltype(K)::value>), grid, dim3(kBlock), 0, st, codes,
                               w.sign, w.level, a);
            return hipGetLastError();
        }
    });
}

hipError_t launch_unpack_dense(const dqgan_plan_s &P, const dqgan_wire &w, float *Phat, hipStream_t st) {
    const RowArgs a = row_args(P, 0.0f, 0);
    const dim3 grid(static_cast<unsigned>(P.n_tiles), static_cast<unsigned>(P.desc.M));
    if (P.desc.kind != kIdentity) {
        hipError_t err = launch_consts_from_scales(P, w.scale, st);
        if (err != hipSuccess) return err;
    }
    return with_dense_kind(P, [&](auto K, auto L) {
        hipLaunchKernelGGL((k_unpack<decltype(K)::value, decltype(L)::value>), grid, dim3(kBlock), 0, st, w.sign,
                           w.level, w.val, Phat, P.d_consts, P.d_off, P.d_tile_seg, a);
        return hipGetLastError();
    });
}

hipError_t launch_aggregate_dense(const dqgan_plan_s &P, const dqgan_wire &w, float *Qhat, hipStream_t st) {
    const RowArgs a = row_args(P, 0.0f, 0);
    const dim3 grid(static_cast<unsigned>((P.n_tiles + kAggQuads - 1) / kAggQuads));  // 16 elements per thread
    const float im = inv_m(P.desc.M);
    if (P.desc.kind != kIdentity) {
        hipError_t err = launch_consts_from_scales(P, w.scale, st);
        if (err != hipSuccess) return err;
    }
    return with_dense_kind(P, [&](auto K, auto L) {
        hipLaunchKernelGGL((k_aggregate<decltype(K)::value, decltype(L)::value>), grid, dim3(kBlock), 0, st, w.sign,
                           w.level, w.val, Qhat, P.d_consts, P.d_off, P.d_tile_seg, a, im);
        return hipGetLastError();
    });
}

hipError_t launch_topk_apply(const dqgan_plan_s &P, float eta, const float *G, float *E, float *W, float *WX,
                             const dqgan_wire &w, float *Qhat, hipStream_t st) {
    const RowArgs a = row_args(P, eta, 0);
    return fused_by_m<kTopk, 0>(P, a, G, E, W, WX, w, Qhat, st);
}

hipError_t launch_topk_encode_rows(const dqgan_plan_s &P, float eta, const float *G, float *E, const dqgan_wire &w,
                                   hipStream_t st) {
    const RowArgs a = row_args(P, eta, 0);
    TopkArgs ta{P.topk.rows, P.topk.tile_off, P.topk.chunk_off, P.topk.n_tiles, P.topk.n_chunks, P.desc.k, w.idx};
    hipLaunchKernelGGL(k_topk_encode_rows, dim3(static_cast<unsigned>(P.topk.n_tiles), static_cast<unsigned>(P.desc.M)),
                       dim3(64), 0, st, G, E, w.val, a, ta);
    return hipGetLastError();
}

hipError_t launch_omd(const dqgan_plan_s &P, float eta, const float *Qhat, float *W, const float *G, const float *E,
                      float *WX, hipStream_t st) {
    hipLaunchKernelGGL(k_omd, dim3(static_cast<unsigned>(P.n_tiles)), dim3(kBlock), 0, st, Qhat, W, G, E, WX, eta,
                       P.desc.d, P.desc.ld, P.desc.M);
    return hipGetLastError();
}

}  // namespace dq
