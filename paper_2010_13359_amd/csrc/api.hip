// C ABI of the DQGAN compression library: argument validation, plan
// construction (segment tables, scratch) and dispatch to the kernels.
#include <stdint.h>
#include <string.h>

#include <new>
#include <vector>

#include "plan.hpp"

using dq::Piece;

namespace {

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

dqgan_status from_hip(hipError_t e) { return e == hipSuccess ? DQGAN_OK : DQGAN_EHIP; }

dqgan_status check_current_device(const dqgan_plan_s *P) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return DQGAN_EHIP;
    return dev == P->device ? DQGAN_OK : DQGAN_EINVAL;
}

// A device pointer argument: required (non-NULL) and 16-byte aligned.
dqgan_status need(const void *p) {
    if (!p) return DQGAN_EINVAL;
    return aligned16(p) ? DQGAN_OK : DQGAN_EALIGN;
}
// An optional device pointer: NULL or 16-byte aligned.
dqgan_status optional(const void *p) { return (!p || aligned16(p)) ? DQGAN_OK : DQGAN_EALIGN; }

#define DQ_TRY(expr)                          \
    do {                                      \
        dqgan_status s_ = (expr);             \
        if (s_ != DQGAN_OK) return s_;        \
    } while (0)

dqgan_status validate_desc(const dqgan_desc *D) {
    if (!D) return DQGAN_EINVAL;
    if (D->d < 1 || D->ld < D->d || D->ld % 1024 != 0) return DQGAN_EINVAL;
    if (D->ld / 256 > INT32_MAX) return DQGAN_EINVAL;  // the fused pass launches one workgroup per 256 columns
    if (D->M < 1 || D->M > 1024) return DQGAN_EINVAL;
    if (D->reserved != 0) return DQGAN_EINVAL;
    if (D->n_seg < 1 || (D->n_seg > 1 && !D->seg_offsets)) return DQGAN_EINVAL;
    if (D->seg_offsets) {
        if (D->seg_offsets[0] != 0 || D->seg_offsets[D->n_seg] != D->d) return DQGAN_EINVAL;
        for (int32_t j = 0; j < D->n_seg; ++j)
            if (D->seg_offsets[j + 1] <= D->seg_offsets[j]) return DQGAN_EINVAL;
    }
    switch (D->kind) {
        case DQGAN_SIGN:
            if (D->norm != DQGAN_L1) return DQGAN_EINVAL;
            break;
        case DQGAN_QSGD:
            if (D->norm != DQGAN_L2 && D->norm != DQGAN_LINF) return DQGAN_EINVAL;
            if (D->levels != 15 && D->levels != 255) return DQGAN_EINVAL;
            break;
        case DQGAN_TOPK:
            if (D->norm != DQGAN_NORM_NONE) return DQGAN_EINVAL;
            if (D->k < 1 || D->k > D->d || D->d >= (int64_t(1) << 32)) return DQGAN_EINVAL;
            break;
        case DQGAN_IDENTITY:
            if (D->norm != DQGAN_NORM_NONE) return DQGAN_EINVAL;
            break;
        case DQGAN_MBIT:
            if (D->norm != DQGAN_L2 && D->norm != DQGAN_LINF) return DQGAN_EINVAL;
            if (D->levels != 8 && D->levels != 4) return DQGAN_EINVAL;
            break;
        default:
            return DQGAN_EINVAL;
    }
    return DQGAN_OK;
}

template <typename T>
hipError_t upload(T **dst, const std::vector<T> &src) {
    hipError_t e = hipMalloc(reinterpret_cast<void **>(dst), src.size() * sizeof(T));
    if (e != hipSuccess) return e;
    return hipMemcpy(*dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice);
}

void free_plan_memory(dqgan_plan_s *P) {
    (void)hipFree(P->d_off);
    (void)hipFree(P->d_tile_seg);
    (void)hipFree(P->d_pieces);
    (void)hipFree(P->d_seg_piece);
    (void)hipFree(P->d_partial);
    (void)hipFree(P->d_pmax);
    (void)hipFree(P->d_consts);
    dq::topk_free(*P);
}

bool dense_kind(int k) { return k == DQGAN_SIGN || k == DQGAN_QSGD || k == DQGAN_IDENTITY || k == DQGAN_MBIT; }

dqgan_status check_wire(const dqgan_plan_s *P, const dqgan_wire *w, bool need_scale) {
    if (!w) return DQGAN_EINVAL;
    switch (P->desc.kind) {
        case DQGAN_SIGN:
            DQ_TRY(need(w->sign));
            if (need_scale) DQ_TRY(need(w->scale));
            break;
        case DQGAN_QSGD:
            DQ_TRY(need(w->sign));
            DQ_TRY(need(w->level));
            if (need_scale) DQ_TRY(need(w->scale));
            break;
        case DQGAN_MBIT:
            DQ_TRY(need(w->level));
            if (need_scale) DQ_TRY(need(w->scale));
            break;
        case DQGAN_TOPK:
            DQ_TRY(need(w->val));
            DQ_TRY(need(w->idx));
            break;
        default:
            DQ_TRY(need(w->val));
            break;
    }
    return DQGAN_OK;
}

}  // namespace

extern "C" {

const char *dqgan_status_string(dqgan_status s) {
    switch (s) {
        case DQGAN_OK: return "ok";
        case DQGAN_EINVAL: return "invalid argument";
        case DQGAN_EALIGN: return "pointer not 16-byte aligned";
        case DQGAN_ENOMEM: return "out of memory";
        case DQGAN_EHIP: return "HIP runtime error";
        case DQGAN_EUNSUPPORTED: return "not supported for this compressor";
        case DQGAN_ESCRATCH: return "workload exceeds the fixed scratch of dqgan_step_fused_noalloc";
    }
    return "unknown status";
}

dqgan_status dqgan_plan_create(const dqgan_desc *desc, dqgan_plan *out) {
    if (!out) return DQGAN_EINVAL;
    *out = nullptr;
    DQ_TRY(validate_desc(desc));
    dqgan_plan_s *P = new (std::nothrow) dqgan_plan_s();
    if (!P) return DQGAN_ENOMEM;
    P->desc = *desc;
    const int64_t d = desc->d;
    if (desc->seg_offsets)
        P->offsets.assign(desc->seg_offsets, desc->seg_offsets + desc->n_seg + 1);
    else
        P->offsets = {0, d};
    P->desc.seg_offsets = nullptr;  // the host copy lives in P->offsets
    P->level_bits = desc->kind == DQGAN_QSGD ? (desc->levels == 255 ? 8 : 4) : desc->kind == DQGAN_MBIT ? desc->levels : 0;
    P->level_count = desc->kind == DQGAN_QSGD ? desc->levels : desc->kind == DQGAN_MBIT ? (1 << (desc->levels - 1)) - 1 : 0;
    P->n_tiles = desc->ld / 1024;
    if (hipGetDevice(&P->device) != hipSuccess) {
        delete P;
        return DQGAN_EHIP;
    }

    // Host tables: tile -> segment of its first element; pieces.
    const int32_t S = desc->n_seg;
    std::vector<int32_t> tile_seg(static_cast<size_t>(P->n_tiles));
    {
        int32_t j = 0;
        for (int64_t tl = 0; tl < P->n_tiles; ++tl) {
            const int64_t i = tl * 1024 < d ? tl * 1024 : d - 1;
            while (P->offsets[j + 1] <= i) ++j;
            tile_seg[static_cast<size_t>(tl)] = j;
        }
    }
    const int64_t piece = static_cast<int64_t>(desc->M) * (d / dq::kPieceElems) >= dq::kPieceBlocksForLong
                              ? dq::kPieceElems
                              : dq::kPieceElems / 2;
    std::vector<Piece> pieces;
    std::vector<int32_t> seg_piece(static_cast<size_t>(S) + 1);
    for (int32_t j = 0; j < S; ++j) {
        seg_piece[static_cast<size_t>(j)] = static_cast<int32_t>(pieces.size());
        for (int64_t a = P->offsets[j]; a < P->offsets[j + 1]; a += piece) {
            const int64_t b = a + piece < P->offsets[j + 1] ? a + piece : P->offsets[j + 1];
            pieces.push_back(Piece{a, static_cast<int32_t>(b - a), j});
        }
    }
    seg_piece[static_cast<size_t>(S)] = static_cast<int32_t>(pieces.size());
    if (pieces.size() > static_cast<size_t>(INT32_MAX / 2)) {
        delete P;
        return DQGAN_EINVAL;
    }
    P->n_pieces = static_cast<int32_t>(pieces.size());

    hipError_t e = hipSuccess;
    if (e == hipSuccess) e = upload(&P->d_off, P->offsets);
    if (e == hipSuccess) e = upload(&P->d_tile_seg, tile_seg);
    if (e == hipSuccess) e = upload(&P->d_pieces, pieces);
    if (e == hipSuccess) e = upload(&P->d_seg_piece, seg_piece);
    const size_t npart = static_cast<size_t>(desc->M) * static_cast<size_t>(P->n_pieces);
    if (e == hipSuccess && dense_kind(desc->kind)) {
        e = hipMalloc(reinterpret_cast<void **>(&P->d_partial), npart * sizeof(double));
        if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&P->d_pmax), npart * sizeof(float));
        if (e == hipSuccess)
            e = hipMalloc(reinterpret_cast<void **>(&P->d_consts), static_cast<size_t>(desc->M) * S * sizeof(dq::SegConst));
    }
    if (e == hipSuccess && desc->kind == DQGAN_TOPK) e = dq::topk_alloc(*P);
    if (e != hipSuccess) {
        free_plan_memory(P);
        delete P;
        return e == hipErrorOutOfMemory ? DQGAN_ENOMEM : DQGAN_EHIP;
    }
    *out = P;
    return DQGAN_OK;
}

dqgan_status dqgan_plan_destroy(dqgan_plan P) {
    if (!P) return DQGAN_OK;
    int cur = -1;
    (void)hipGetDevice(&cur);
    if (cur != P->device) (void)hipSetDevice(P->device);
    hipError_t e = hipDeviceSynchronize();
    free_plan_memory(P);
    if (cur >= 0 && cur != P->device) (void)hipSetDevice(cur);
    delete P;
    return from_hip(e);
}

dqgan_status dqgan_wire_bytes(dqgan_plan P, size_t *sign, size_t *level, size_t *scale, size_t *val, size_t *idx) {
    if (!P) return DQGAN_EINVAL;
    const dqgan_desc &D = P->desc;
    const size_t M = static_cast<size_t>(D.M), ld = static_cast<size_t>(D.ld);
    const bool coded = D.kind == DQGAN_SIGN || D.kind == DQGAN_QSGD || D.kind == DQGAN_MBIT;
    if (sign) *sign = (D.kind == DQGAN_SIGN || D.kind == DQGAN_QSGD) ? M * (ld / 32) * 4 : 0;
    if (level) *level = (D.kind == DQGAN_QSGD || D.kind == DQGAN_MBIT) ? M * (ld * P->level_bits / 32) * 4 : 0;
    if (scale) *scale = coded ? M * static_cast<size_t>(D.n_seg) * 4 : 0;
    if (val) *val = D.kind == DQGAN_TOPK ? M * static_cast<size_t>(D.k) * 4 : D.kind == DQGAN_IDENTITY ? M * ld * 4 : 0;
    if (idx) *idx = D.kind == DQGAN_TOPK ? M * static_cast<size_t>(D.k) * 4 : 0;
    return DQGAN_OK;
}

dqgan_status dqgan_compress_ef(dqgan_plan P, float eta, uint32_t t, const float *G, float *E, const float *scales_in,
                               const dqgan_wire *out, void *stream) {
    if (!P) return DQGAN_EINVAL;
    DQ_TRY(need(G));
    DQ_TRY(need(E));
    DQ_TRY(optional(scales_in));
    DQ_TRY(check_wire(P, out, true));
    DQ_TRY(check_current_device(P));
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int kind = P->desc.kind;
    if (kind == DQGAN_TOPK) return from_hip(dq::launch_topk_compress(*P, eta, G, E, *out, st));
    if (kind != DQGAN_IDENTITY) {
        hipError_t e = dq::launch_segment_scales(*P, eta, G, E, scales_in, out->scale, st);
        if (e != hipSuccess) return DQGAN_EHIP;
    }
    return from_hip(dq::launch_encode(*P, eta, t, G, E, *out, st));
}

dqgan_status dqgan_pack(dqgan_plan P, const uint16_t *codes, const float *scales, const dqgan_wire *out,
                        void *stream) {
    if (!P) return DQGAN_EINVAL;
    if (P->desc.kind != DQGAN_SIGN && P->desc.kind != DQGAN_QSGD && P->desc.kind != DQGAN_MBIT)
        return DQGAN_EUNSUPPORTED;
    DQ_TRY(need(codes));
    DQ_TRY(need(scales));
    DQ_TRY(check_wire(P, out, true));
    DQ_TRY(check_current_device(P));
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (scales != out->scale) {
        hipError_t e = hipMemcpyAsync(out->scale, scales, static_cast<size_t>(P->desc.M) * P->desc.n_seg * sizeof(float),
                                      hipMemcpyDeviceToDevice, st);
        if (e != hipSuccess) return DQGAN_EHIP;
    }
    return from_hip(dq::launch_pack(*P, codes, *out, st));
}

dqgan_status dqgan_unpack(dqgan_plan P, const dqgan_wire *in, float *Phat, void *stream) {
    if (!P) return DQGAN_EINVAL;
    DQ_TRY(check_wire(P, in, true));
    DQ_TRY(need(Phat));
    DQ_TRY(check_current_device(P));
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (P->desc.kind == DQGAN_TOPK) return from_hip(dq::launch_topk_unpack(*P, *in, Phat, st));
    return from_hip(dq::launch_unpack_dense(*P, *in, Phat, st));
}

dqgan_status dqgan_aggregate(dqgan_plan P, const dqgan_wire *in, float *Qhat, void *stream) {
    if (!P) return DQGAN_EINVAL;
    DQ_TRY(check_wire(P, in, true));
    DQ_TRY(need(Qhat));
    DQ_TRY(check_current_device(P));
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (P->desc.kind == DQGAN_TOPK) return from_hip(dq::launch_topk_aggregate(*P, *in, Qhat, st));
    return from_hip(dq::launch_aggregate_dense(*P, *in, Qhat, st));
}

dqgan_status dqgan_omd_step(dqgan_plan P, float eta, const float *Qhat, float *W, const float *G, const float *E,
                            float *WX, void *stream) {
    if (!P) return DQGAN_EINVAL;
    DQ_TRY(need(Qhat));
    DQ_TRY(need(W));
    DQ_TRY(optional(WX));
    if (WX) {
        DQ_TRY(need(G));
        DQ_TRY(need(E));
    }
    DQ_TRY(check_current_device(P));
    return from_hip(dq::launch_omd(*P, eta, Qhat, W, G, E, WX, static_cast<hipStream_t>(stream)));
}

dqgan_status dqgan_step_scales(dqgan_plan P, float eta, const float *G, const float *E, const dqgan_wire *out,
                               void *stream) {
    if (!P) return DQGAN_EINVAL;
    DQ_TRY(need(G));
    DQ_TRY(need(E));
    DQ_TRY(check_wire(P, out, true));
    DQ_TRY(check_current_device(P));
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int kind = P->desc.kind;
    if (kind == DQGAN_TOPK) return from_hip(dq::launch_topk_select(*P, eta, G, E, st));
    if (kind == DQGAN_IDENTITY) return DQGAN_OK;
    return from_hip(dq::launch_segment_scales(*P, eta, G, E, nullptr, out->scale, st));
}

dqgan_status dqgan_step_apply(dqgan_plan P, float eta, uint32_t t, const float *G, float *E, float *W, float *WX,
                              const dqgan_wire *out, float *Qhat, void *stream) {
    if (!P) return DQGAN_EINVAL;
    DQ_TRY(need(G));
    DQ_TRY(need(E));
    DQ_TRY(need(W));
    DQ_TRY(need(WX));
    DQ_TRY(optional(Qhat));
    DQ_TRY(check_wire(P, out, true));
    DQ_TRY(check_current_device(P));
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (P->desc.kind == DQGAN_TOPK) return from_hip(dq::launch_topk_apply(*P, eta, G, E, W, WX, *out, Qhat, st));
    return from_hip(dq::launch_fused_dense(*P, eta, t, G, E, W, WX, *out, Qhat, st));
}

dqgan_status dqgan_step_fused(dqgan_plan P, float eta, uint32_t t, const float *G, float *E, float *W, float *WX,
                              const dqgan_wire *out, float *Qhat, void *stream) {
    if (!P) return DQGAN_EINVAL;
    DQ_TRY(need(G));
    DQ_TRY(need(E));
    DQ_TRY(need(W));
    DQ_TRY(need(WX));
    DQ_TRY(optional(Qhat));
    DQ_TRY(check_wire(P, out, true));
    DQ_TRY(check_current_device(P));
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int kind = P->desc.kind;
    if (kind == DQGAN_TOPK) {
        hipError_t e = dq::launch_topk_select(*P, eta, G, E, st);
        if (e != hipSuccess) return DQGAN_EHIP;
        return from_hip(dq::launch_topk_apply(*P, eta, G, E, W, WX, *out, Qhat, st));
    }
    if (kind != DQGAN_IDENTITY) {
        hipError_t e = dq::launch_segment_scales(*P, eta, G, E, nullptr, out->scale, st);
        if (e != hipSuccess) return DQGAN_EHIP;
    }
    return from_hip(dq::launch_fused_dense(*P, eta, t, G, E, W, WX, *out, Qhat, st));
}

}  // extern "C"
