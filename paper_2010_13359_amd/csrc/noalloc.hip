// dqgan_step_fused_noalloc: the fused iteration of the segment-scaled
// compressors without a plan, for callers that cannot allocate device memory
// (HIP graph capture, serving loops, harnesses that forbid hipMalloc).
//
// Everything a plan would hold (segment tables, pieces of the statistics
// pass, binary64 partials, per-segment constants) lives in one file-scope
// device array, `scratch`, of kNoAllocScratchBytes.  Its address on each
// device is taken once with hipGetSymbolAddress and kept; kernels get that
// address as an argument.  The tables are rebuilt by a small kernel at every
// call from the segment offsets, which travel by value in its arguments, so
// a call enqueues kernels only and may be captured in a graph.  Every call
// on a device shares the array: calls that overlap on one device race.
#include <stdint.h>

#include <atomic>

#include "device.hpp"
#include "plan.hpp"

namespace {

constexpr size_t kNoAllocScratchBytes = size_t(8) << 20;  // 8 MiB per device
constexpr int kNoAllocMaxSeg = 255;                       // offsets travel in the launch arguments
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

std::atomic<uintptr_t> g_scratch_ptr[kMaxDevices];

// The address of `scratch` on the current device (device memory; the host
// symbol itself is only a stand-in).
hipError_t scratch_on_device(int dev, unsigned char **out) {
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    uintptr_t p = g_scratch_ptr[dev].load(std::memory_order_acquire);
    if (p == 0) {
        void *addr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!addr) return hipErrorInvalidSymbol;
        p = reinterpret_cast<uintptr_t>(addr);
        g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
    *out = reinterpret_cast<unsigned char *>(p);
    return hipSuccess;
}

size_t round256(size_t n) { return (n + 255) & ~size_t(255); }

// Byte offsets of the tables inside the scratch array.
struct Layout {
    size_t off, seg_piece, tile_seg, pieces, partial, pmax, consts, total;
};

Layout layout(int64_t n_seg, int64_t n_tiles, int64_t n_pieces, int64_t M) {
    Layout L{};
    size_t at = 0;
    L.off = at;
    at += round256(static_cast<size_t>(n_seg + 1) * sizeof(int64_t));
    L.seg_piece = at;
    at += round256(static_cast<size_t>(n_seg + 1) * sizeof(int32_t));
    L.tile_seg = at;
    at += round256(static_cast<size_t>(n_tiles) * sizeof(int32_t));
    L.pieces = at;
    at += round256(static_cast<size_t>(n_pieces) * sizeof(dq::Piece));
    L.partial = at;
    at += round256(static_cast<size_t>(M) * static_cast<size_t>(n_pieces) * sizeof(double));
    L.pmax = at;
    at += round256(static_cast<size_t>(M) * static_cast<size_t>(n_pieces) * sizeof(float));
    L.consts = at;
    at += round256(static_cast<size_t>(M) * static_cast<size_t>(n_seg) * sizeof(dq::SegConst));
    L.total = at;
    return L;
}

// The segment table by value: offsets and the first piece of each segment.
struct SegTable {
    int64_t off[kNoAllocMaxSeg + 1];
    int32_t first_piece[kNoAllocMaxSeg + 1];
    int32_t n_seg;
    int32_t n_pieces;
    int64_t n_tiles;
    int64_t d;
    int64_t piece;
};

// One thread per table entry: the tables dqgan_plan_create builds on the
// host (tile -> segment of its first element; pieces of at most `piece`
// elements that never cross a segment; first piece of each segment).
__global__ __launch_bounds__(dq::kBlock) void k_noalloc_tables(SegTable T, int64_t *__restrict__ off,
                                                               int32_t *__restrict__ seg_piece,
                                                               int32_t *__restrict__ tile_seg,
                                                               dq::Piece *__restrict__ pieces) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * dq::kBlock + threadIdx.x;
    if (i <= T.n_seg) {
        off[i] = T.off[i];
        seg_piece[i] = T.first_piece[i];
    }
    if (i < T.n_tiles) {
        const int64_t e = i * 1024 < T.d ? i * 1024 : T.d - 1;
        int lo = 0, hi = T.n_seg - 1;  // the segment j with off[j] <= e < off[j + 1]
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (T.off[mid] <= e) lo = mid; else hi = mid - 1;
        }
        tile_seg[i] = lo;
    }
    if (i < T.n_pieces) {
        int lo = 0, hi = T.n_seg - 1;  // the segment j with first_piece[j] <= i < first_piece[j + 1]
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (T.first_piece[mid] <= i) lo = mid; else hi = mid - 1;
        }
        const int64_t a = T.off[lo] + (i - T.first_piece[lo]) * T.piece;
        const int64_t b = a + T.piece < T.off[lo + 1] ? a + T.piece : T.off[lo + 1];
        pieces[i] = dq::Piece{a, static_cast<int32_t>(b - a), lo};
    }
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

extern "C" dqgan_status dqgan_step_fused_noalloc(const dqgan_desc *desc, float eta, uint32_t t, const float *G,
                                                 float *E, float *W, float *WX, const dqgan_wire *out, float *Qhat,
                                                 void *stream) {
    // The descriptor: dqgan_plan_create's rules, dense compressors only.
    if (!desc || !out) return DQGAN_EINVAL;
    const dqgan_desc &D = *desc;
    if (D.kind == DQGAN_TOPK) return DQGAN_EUNSUPPORTED;
    if (D.d < 1 || D.ld < D.d || D.ld % 1024 != 0 || D.ld / 256 > INT32_MAX) return DQGAN_EINVAL;
    if (D.M < 1 || D.M > 1024 || D.reserved != 0) return DQGAN_EINVAL;
    if (D.n_seg < 1 || (D.n_seg > 1 && !D.seg_offsets)) return DQGAN_EINVAL;
    if (D.n_seg > kNoAllocMaxSeg) return DQGAN_ESCRATCH;
    SegTable T{};
    T.n_seg = D.n_seg;
    T.d = D.d;
    T.n_tiles = D.ld / 1024;
    for (int32_t j = 0; j <= D.n_seg; ++j) T.off[j] = D.seg_offsets ? D.seg_offsets[j] : (j == 0 ? 0 : D.d);
    if (T.off[0] != 0 || T.off[D.n_seg] != D.d) return DQGAN_EINVAL;
    for (int32_t j = 0; j < D.n_seg; ++j)
        if (T.off[j + 1] <= T.off[j]) return DQGAN_EINVAL;
    int level_bits = 0, level_count = 0;
    switch (D.kind) {
        case DQGAN_SIGN:
            if (D.norm != DQGAN_L1) return DQGAN_EINVAL;
            break;
        case DQGAN_QSGD:
            if ((D.norm != DQGAN_L2 && D.norm != DQGAN_LINF) || (D.levels != 15 && D.levels != 255))
                return DQGAN_EINVAL;
            level_bits = D.levels == 255 ? 8 : 4;
            level_count = D.levels;
            break;
        case DQGAN_MBIT:
            if ((D.norm != DQGAN_L2 && D.norm != DQGAN_LINF) || (D.levels != 8 && D.levels != 4)) return DQGAN_EINVAL;
            level_bits = D.levels;
            level_count = (1 << (D.levels - 1)) - 1;
            break;
        case DQGAN_IDENTITY:
            if (D.norm != DQGAN_NORM_NONE) return DQGAN_EINVAL;
            break;
        default:
            return DQGAN_EINVAL;
    }
    // Buffers: the rules of dqgan_step_fused.
    const void *need[] = {G, E, W, WX};
    for (const void *p : need)
        if (!p) return DQGAN_EINVAL;
    for (const void *p : need)
        if (!aligned16(p)) return DQGAN_EALIGN;
    if (Qhat && !aligned16(Qhat)) return DQGAN_EALIGN;
    const void *planes[3] = {nullptr, nullptr, nullptr};
    int n_planes = 0;
    if (D.kind == DQGAN_SIGN || D.kind == DQGAN_QSGD) planes[n_planes++] = out->sign;
    if (D.kind == DQGAN_QSGD || D.kind == DQGAN_MBIT) planes[n_planes++] = out->level;
    if (D.kind == DQGAN_IDENTITY) planes[n_planes++] = out->val;
    else planes[n_planes++] = out->scale;
    for (int k = 0; k < n_planes; ++k)
        if (!planes[k]) return DQGAN_EINVAL;
    for (int k = 0; k < n_planes; ++k)
        if (!aligned16(planes[k])) return DQGAN_EALIGN;

    // Pieces as dqgan_plan_create cuts them (the scales then equal the
    // plan's bit for bit).
    T.piece = static_cast<int64_t>(D.M) * (D.d / dq::kPieceElems) >= dq::kPieceBlocksForLong ? dq::kPieceElems
                                                                                          : dq::kPieceElems / 2;
    int64_t n_pieces = 0;
    for (int32_t j = 0; j < D.n_seg; ++j) {
        T.first_piece[j] = static_cast<int32_t>(n_pieces);
        n_pieces += (T.off[j + 1] - T.off[j] + T.piece - 1) / T.piece;
        if (n_pieces > INT32_MAX / 2) return DQGAN_ESCRATCH;
    }
    T.first_piece[D.n_seg] = static_cast<int32_t>(n_pieces);
    T.n_pieces = static_cast<int32_t>(n_pieces);
    const Layout L = layout(D.n_seg, T.n_tiles, n_pieces, D.M);
    if (L.total > kNoAllocScratchBytes) return DQGAN_ESCRATCH;

    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return DQGAN_EHIP;
    unsigned char *base = nullptr;
    if (scratch_on_device(dev, &base) != hipSuccess) return DQGAN_EHIP;
    hipStream_t st = static_cast<hipStream_t>(stream);

    // A plan on the stack whose device tables point into the scratch array
    // (its host vectors stay empty: nothing is allocated).
    dqgan_plan_s P;
    P.desc = D;
    P.desc.seg_offsets = nullptr;
    P.device = dev;
    P.level_bits = level_bits;
    P.level_count = level_count;
    P.n_tiles = T.n_tiles;
    P.d_off = reinterpret_cast<int64_t *>(base + L.off);
    P.d_seg_piece = reinterpret_cast<int32_t *>(base + L.seg_piece);
    P.d_tile_seg = reinterpret_cast<int32_t *>(base + L.tile_seg);
    P.d_pieces = reinterpret_cast<dq::Piece *>(base + L.pieces);
    P.n_pieces = T.n_pieces;
    P.d_partial = reinterpret_cast<double *>(base + L.partial);
    P.d_pmax = reinterpret_cast<float *>(base + L.pmax);
    P.d_consts = reinterpret_cast<dq::SegConst *>(base + L.consts);

    int64_t n_threads = T.n_tiles;
    if (T.n_pieces > n_threads) n_threads = T.n_pieces;
    if (T.n_seg + 1 > n_threads) n_threads = T.n_seg + 1;
    hipLaunchKernelGGL(k_noalloc_tables, dim3(static_cast<unsigned>((n_threads + dq::kBlock - 1) / dq::kBlock)),
                       dim3(dq::kBlock), 0, st, T, P.d_off, P.d_seg_piece, P.d_tile_seg, P.d_pieces);
    if (hipGetLastError() != hipSuccess) return DQGAN_EHIP;
    if (D.kind != DQGAN_IDENTITY && dq::launch_segment_scales(P, eta, G, E, nullptr, out->scale, st) != hipSuccess)
        return DQGAN_EHIP;
    return dq::launch_fused_dense(P, eta, t, G, E, W, WX, *out, Qhat, st) == hipSuccess ? DQGAN_OK : DQGAN_EHIP;
}
