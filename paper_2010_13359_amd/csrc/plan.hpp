// Plan object and internal launchers of the DQGAN library (host side).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "../../include/dqgan.h"

namespace dq {

// A contiguous run of one segment of a row, at most kPieceElems long; the
// norm pass reduces one piece per workgroup.  Pieces never cross segments.
struct Piece {
    int64_t start;
    int32_t len;
    int32_t seg;
};
constexpr int64_t kPieceElems = 16384;

// Top-k workspace (one set per plan).
struct TopkScratch {
    uint32_t *hist = nullptr;       // [M][kHistBins] counts of the current digit
    uint32_t *state = nullptr;      // [M][kTopkState] selection state per row
    uint32_t *tile_cnt = nullptr;   // [M][n_tiles] selected elements per tile
    uint32_t *tile_off = nullptr;   // [M][n_tiles] exclusive prefix of tile_cnt
    int64_t n_tiles = 0;
};

}  // namespace dq

struct dqgan_plan_s {
    dqgan_desc desc{};
    std::vector<int64_t> offsets;  // host copy, n_seg + 1
    int device = 0;
    int level_bits = 0;            // QSGD: 8 (s = 255) or 4 (s = 15)
    int64_t n_tiles = 0;           // ld / 1024

    int64_t *d_off = nullptr;       // [n_seg + 1]
    int32_t *d_tile_seg = nullptr;  // [n_tiles] segment of each tile's first element
    dq::Piece *d_pieces = nullptr;  // [n_pieces]
    int32_t n_pieces = 0;
    int32_t *d_seg_piece = nullptr;  // [n_seg + 1] first piece of each segment
    double *d_partial = nullptr;     // [M][n_pieces] partial sums (L1, L2^2)
    float *d_pmax = nullptr;         // [M][n_pieces] partial maxima (Linf)
    float2 *d_consts = nullptr;      // [M][n_seg] per-segment constants
    dq::TopkScratch topk;
};

namespace dq {

// Dense compressors (SIGN, QSGD, IDENTITY).
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
hipError_t launch_topk_unpack(const dqgan_plan_s &P, const dqgan_wire &w, float *Phat, hipStream_t st);
hipError_t launch_topk_aggregate(const dqgan_plan_s &P, const dqgan_wire &w, float *Qhat, hipStream_t st);

}  // namespace dq
