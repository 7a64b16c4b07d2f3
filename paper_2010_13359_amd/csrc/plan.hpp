// Plan object and internal launchers of the DQGAN library (host side).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "../../include/dqgan.h"

namespace dq {

// A contiguous run of one segment of a row, at most kPieceElems long (half
// that for workloads with few pieces); the norm pass reduces one piece per
// workgroup.  Pieces never cross segments.
struct Piece {
    int64_t start;
    int32_t len;
    int32_t seg;
};
constexpr int64_t kPieceElems = 32768;
// Below this many (worker, piece) workgroups the pieces are halved: the
// statistics pass over 32 workers x 2^25 elements ran 1.5 % faster with
// 32768-element pieces than with 16384, over 16 workers x 6.3M elements 2 %
// slower.
constexpr int64_t kPieceBlocksForLong = 16384;

// Per (worker, segment) constants of the segment-scaled compressors.
// SIGN: a = the scale.  QSGD, MBIT (equation qsgd): a = fl(s / (u sigma))
// and b = fl(u sigma / s), where u = 2^64 for sigma < 2^-64 (so that s / sigma
// cannot overflow binary32 and sigma / s keeps its significand) and u = 1
// otherwise; with u = 2^64 both are stored negated, and the kernels then
// multiply |p| by 2^64 before the product with |a| and the decoded magnitude
// fl(level * |b|) by 2^-64.  A norm of 0 or one that is not finite gives
// a = b = 0: level 0 everywhere.
struct alignas(8) SegConst {
    float a, b;
};

// Capacity of the MI355X Infinity Cache (memory-side, in front of HBM): the
// fused pass streams message planes larger than this past the caches.
constexpr double kInfinityCacheBytes = 256.0 * 1024 * 1024;

// Per-worker selection state of the top-k compressor.  Keys are the binary32
// bit patterns of |p| (monotone in |p|).  Element i is selected iff
// key > T, or key == T and i <= I.
struct TopkRow {
    uint32_t lo, hi;     // candidate band [lo, hi] of keys, from the sample
    uint32_t n_cand;     // candidates staged into the row's list by the full pass (may exceed the capacity);
                         // this and n_spill, n_above are counted in TopkScratch::ctr and copied here
    uint32_t fallback;   // 1: the band missed the k-th key; the full-row search decides
    uint32_t T, I;       // the selection
    uint32_t n_spill;    // candidates a wave could not stage: stored from the top of the row's list down
    uint32_t slots;      // bit p: the candidate search built digit histogram p in this iteration
    uint32_t pad1;
    uint32_t pad0;
    uint32_t total;      // selected count found by the tile scan (equals k)
    uint32_t n_above;    // keys above the band, counted by the full pass
    uint32_t pad[4];
};

constexpr int kTopkTile = 256;            // elements per counting tile (one wave of quads)
// The counters that many workgroups of one kernel update atomically live in
// their own block of TopkScratch::ctr, not in the row's TopkRow: every
// workgroup of the full pass reads its row's band from rows[m] when it
// starts, and the other workgroups' atomics on the same cache line held the
// pass 0.3 ms back at 64 rows of 10^8.  The first search kernel copies the
// pass's counters into rows[m]; the finish reads the play count here.
constexpr int kRowCtrWords = 64;          // words per row (one 256-byte block)
constexpr int kCtrCand = 0, kCtrAbove = 1, kCtrSpill = 2;
constexpr int kCtrPlay = 3;  // candidates still in play after the first key digit, listed for the finish
constexpr int kTopkChunkTiles = 64;       // tiles per workgroup of the full pass: one candidate run each
constexpr int kSampleBins = 32768;        // sample histogram: key >> 16 (keys < 2^31)
constexpr int64_t kSampleStride = 65536;  // one 256-element chunk sampled per 65536 elements
constexpr int kDigitBins = 2048;          // radix-select histograms: 11-bit digits
constexpr int kSelectPasses = 6;          // histogram slots of a search: up to 3 key digits, 3 index digits

// Top-k workspace (one set per plan).
struct TopkScratch {
    TopkRow *rows = nullptr;        // [M]
    uint32_t *ctr = nullptr;        // [M][kRowCtrWords] the full pass's counters of each row, apart from rows
    uint32_t *hist = nullptr;       // [M][kSampleBins] sample histogram (zero between iterations)
    uint32_t *sel_hist = nullptr;   // [M][kDigitBins] histogram of the first key digit among the candidates
    uint2 *play = nullptr;          // [M][cap] the candidates in play after the first key digit
    uint32_t *fb_hist = nullptr;    // [M][kSelectPasses][kDigitBins] digit histograms of the full-row search
    uint2 *cand = nullptr;          // [M][cap] (key, index) candidates: runs from the bottom, spills from the top
    int64_t cap = 0;
    uint2 *runs = nullptr;          // [M][n_chunks] (first position, count) of each full-pass workgroup's candidates
    uint16_t *tile_cnt = nullptr;   // [M][n_tiles] selected elements per 256-element tile (at most 256)
    uint16_t *tile_off = nullptr;   // [M][n_tiles] selected elements before the tile within its chunk (< 2^14)
    uint32_t *chunk_sum = nullptr;  // [M][n_chunks] selected elements per chunk of kTopkChunkTiles tiles
    uint32_t *chunk_off = nullptr;  // [M][n_chunks] exclusive prefix of chunk_sum
    uint32_t *agg_start = nullptr;  // [n_agg_tiles + 1][M] first message entry per server-average tile
    int64_t n_agg_tiles = 0;
    int64_t n_tiles = 0;
    int64_t n_chunks = 0;           // chunks of kTopkChunkTiles tiles per row
    int64_t n_sample_chunks = 0;    // sampled chunks per row
    uint32_t n_samples = 0;         // sampled elements per row
};

// The state the apply pass reads: the threshold per row and each tile's
// first output position, tile_off + chunk_off of its chunk.
struct TopkArgs {
    const TopkRow *rows;
    const uint16_t *tile_off;
    const uint32_t *chunk_off;
    int64_t n_tiles;
    int64_t n_chunks;
    int64_t k;
    uint32_t *idx;
};

__device__ __forceinline__ uint32_t topk_tile_base(const TopkArgs &ta, int m, int64_t tile) {
    return ta.tile_off[static_cast<int64_t>(m) * ta.n_tiles + tile] +
           ta.chunk_off[static_cast<int64_t>(m) * ta.n_chunks + tile / kTopkChunkTiles];
}

}  // namespace dq

struct dqgan_plan_s {
    dqgan_desc desc{};
    std::vector<int64_t> offsets;  // host copy, n_seg + 1
    int device = 0;
    int level_bits = 0;            // QSGD: 8 (s = 255) or 4 (s = 15); MBIT: m
    int level_count = 0;           // quantizer levels: QSGD s; MBIT k = 2^(m-1) - 1
    int64_t n_tiles = 0;           // ld / 1024

    int64_t *d_off = nullptr;       // [n_seg + 1]
    int32_t *d_tile_seg = nullptr;  // [n_tiles] segment of each tile's first element
    dq::Piece *d_pieces = nullptr;  // [n_pieces]
    int32_t n_pieces = 0;
    int32_t *d_seg_piece = nullptr;  // [n_seg + 1] first piece of each segment
    double *d_partial = nullptr;     // [M][n_pieces] partial sums (L1, L2^2)
    float *d_pmax = nullptr;         // [M][n_pieces] partial maxima (Linf)
    dq::SegConst *d_consts = nullptr;  // [M][n_seg] per-segment constants
    dq::TopkScratch topk;
};

namespace dq {

// Dense compressors (SIGN, QSGD, MBIT, IDENTITY).
hipError_t launch_segment_scales(const dqgan_plan_s &P, float eta, const float *G, const float *E,
                                 const float *scales_in, float *scale_out, hipStream_t st);
hipError_t launch_consts_from_scales(const dqgan_plan_s &P, const float *scales, hipStream_t st);
hipError_t launch_encode(const dqgan_plan_s &P, float eta, uint32_t t, const float *G, float *E,
                         const dqgan_wire &w, hipStream_t st);
hipError_t launch_fused_dense(const dqgan_plan_s &P, float eta, uint32_t t, const float *G, float *E, float *W,
                              float *WX, const dqgan_wire &w, float *Qhat, hipStream_t st);
hipError_t launch_pack(const dqgan_plan_s &P, const uint16_t *codes, const dqgan_wire &w, hipStream_t st);
hipError_t launch_unpack_dense(const dqgan_plan_s &P, const dqgan_wire &w, float *Phat, hipStream_t st);
hipError_t launch_aggregate_dense(const dqgan_plan_s &P, const dqgan_wire &w, float *Qhat, hipStream_t st);
hipError_t launch_omd(const dqgan_plan_s &P, float eta, const float *Qhat, float *W, const float *G,
                      const float *E, float *WX, hipStream_t st);

// Top-k.
hipError_t topk_alloc(dqgan_plan_s &P);
void topk_free(dqgan_plan_s &P);
hipError_t launch_topk_compress(const dqgan_plan_s &P, float eta, const float *G, float *E, const dqgan_wire &w,
                                hipStream_t st);
hipError_t launch_topk_select(const dqgan_plan_s &P, float eta, const float *G, const float *E, hipStream_t st);
hipError_t launch_topk_apply(const dqgan_plan_s &P, float eta, const float *G, float *E, float *W, float *WX,
                             const dqgan_wire &w, float *Qhat, hipStream_t st);
hipError_t launch_topk_encode_rows(const dqgan_plan_s &P, float eta, const float *G, float *E, const dqgan_wire &w,
                                   hipStream_t st);
hipError_t launch_topk_unpack(const dqgan_plan_s &P, const dqgan_wire &w, float *Phat, hipStream_t st);
hipError_t launch_topk_aggregate(const dqgan_plan_s &P, const dqgan_wire &w, float *Qhat, hipStream_t st);

}  // namespace dq
