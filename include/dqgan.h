/*
 * dqgan.h -- C ABI of the MI355X (gfx950) library for the per-iteration
 * gradient-compression path of DQGAN (Chen, Yang, Shen, Pang, "A Distributed
 * Training Algorithm of Generative Adversarial Networks with Quantized
 * Gradients", arXiv:2010.13359, Algorithm 2).
 *
 * One iteration t of Algorithm 2, for M workers whose vectors are the M rows
 * of one matrix in device memory:
 *   worker m:  p_t = eta * g_t + e_{t-1}            (EF accumulate)
 *              p-hat_t = Q(p_t), pushed to server   (compress + pack)
 *              e_t = p_t - p-hat_t                  (EF residual)
 *   server:    q-hat_t = (1/M) sum_m p-hat_t^(m)    (unpack + average)
 *   worker m:  w_t = w_{t-1} - q-hat_t              (OMD update)
 *              w_{t+1/2}^(m) = w_t - (eta g_t + e_t)  (the next evaluation
 *              point: the first worker step of iteration t+1, which reuses
 *              the stored gradient and compensates the error a second time)
 *
 * Conventions shared by every call:
 *  - Matrices G (gradients), E (error residuals), WX (evaluation points) and
 *    P-hat are row-major fp32 [M][ld]; row m starts at element m*ld.  ld is a
 *    multiple of 1024 and ld >= d.  Vectors W and Q-hat hold ld floats.
 *    Elements [d, ld) of a row are padding: never read into a result.  The
 *    padding of E and W is preserved, that of WX, P-hat and Q-hat is written
 *    as 0, and message bits beyond d are 0.
 *  - Every pointer is a device pointer (hipMalloc'd or equivalent), 16-byte
 *    aligned, owned by the caller, except those marked "host".  The buffers
 *    of one call must not overlap (E is updated in place; G, E, W, WX, Qhat,
 *    P-hat and the message planes are distinct).
 *  - Arithmetic is IEEE binary32 with round-to-nearest-even, one rounding per
 *    operation, no fused multiply-add where the definitions below list
 *    separate operations; segment norms are summed in binary64 and rounded
 *    once.
 *  - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *    stream).  Arguments are validated synchronously before anything is
 *    enqueued; an invalid argument returns an error code and enqueues
 *    nothing.  A failed launch returns DQGAN_EHIP; faults of enqueued work
 *    surface at the caller's next synchronization.  No call aborts the
 *    process.  Only dqgan_plan_create and dqgan_plan_destroy allocate or free
 *    device memory.  The per-iteration calls enqueue kernels only (plus, in
 *    dqgan_pack, one device-to-device copy of the scales): no memset, no host
 *    synchronization, so a caller may capture them in a HIP graph and replay
 *    it.
 *  - A plan is bound to the device that was current at its creation; calls
 *    must be made with that device current.  A plan is not thread-safe, and
 *    two calls on one plan must not run concurrently on different streams
 *    (they share the plan's scratch).  Distinct plans are independent.
 */
#ifndef DQGAN_H
#define DQGAN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DQGAN_OK = 0,
    DQGAN_EINVAL = -1,       /* invalid argument (size, kind, NULL pointer) */
    DQGAN_EALIGN = -2,       /* a pointer is not 16-byte aligned            */
    DQGAN_ENOMEM = -3,       /* device or host allocation failed             */
    DQGAN_EHIP = -4,         /* a HIP runtime call or launch failed          */
    DQGAN_EUNSUPPORTED = -5, /* valid, but not offered for this compressor   */
    DQGAN_ESCRATCH = -6      /* the workload exceeds the fixed scratch of
                                dqgan_step_fused_noalloc                     */
} dqgan_status;

/* The delta-approximate compressors Q (Definition 1). */
typedef enum {
    DQGAN_SIGN = 0,     /* scaled sign: one scale per (worker, segment)
                           (Section 2.4, sign with a scaling factor)         */
    DQGAN_QSGD = 1,     /* s-level stochastic quantizer, equation (qsgd)    */
    DQGAN_TOPK = 2,     /* k largest magnitudes (Theorem 1)                 */
    DQGAN_IDENTITY = 3, /* Q = id (delta = 1): the uncompressed special case */
    DQGAN_MBIT = 4      /* m-bit sign-magnitude stochastic quantizer with
                           k = 2^(m-1) - 1 uniform levels (Appendix A); with
                           DQGAN_LINF the compressor of the experiments     */
} dqgan_kind;

typedef enum {
    DQGAN_NORM_NONE = 0,
    DQGAN_L1 = 1,       /* SIGN: scale = ||p_seg||_1 / n_seg                  */
    DQGAN_L2 = 2,       /* QSGD: sigma = ||p_seg||_2, equation (qsgd)         */
    DQGAN_LINF = 3      /* QSGD: sigma = ||p_seg||_inf (Hou et al. variant)   */
} dqgan_norm;

typedef struct {
    int64_t d;                    /* parameters per worker, d >= 1                 */
    int64_t ld;                   /* row stride: ld >= d, ld % 1024 == 0,
                                     ld / 256 <= 2^31 - 1                          */
    int32_t M;                    /* workers, 1 <= M <= 1024                        */
    int32_t n_seg;                /* segments (SIGN, QSGD); 1 for the others        */
    const int64_t *seg_offsets;   /* host, n_seg + 1 entries, strictly increasing,
                                     seg_offsets[0] = 0, seg_offsets[n_seg] = d;
                                     copied by dqgan_plan_create                   */
    int32_t kind;                 /* dqgan_kind                                     */
    int32_t norm;                 /* SIGN: DQGAN_L1; QSGD, MBIT: DQGAN_L2 or
                                     DQGAN_LINF; TOPK, IDENTITY: DQGAN_NORM_NONE   */
    int32_t levels;               /* QSGD s: 255 (8-bit level field) or 15 (4-bit);
                                     MBIT: code bits m, 8 or 4 (k = 127 or 7)      */
    int32_t reserved;             /* must be 0                                      */
    int64_t k;                    /* TOPK: 1 <= k <= d, d < 2^32                    */
    uint64_t seed;                /* QSGD, MBIT: key of the Philox4x32-10 generator */
} dqgan_desc;

typedef struct dqgan_plan_s *dqgan_plan;

/* The message each worker pushes to the server (Algorithm 2), all M rows.
 * Sign plane (SIGN, QSGD): uint32 [M][ld/32]; element i of a row is bit
 *   (i & 31) of word i >> 5; 1 means the sign bit of p_i is set.
 * Level plane (QSGD): uint32 [M][ld*b/32] with b = 8 (s = 255) or 4 (s = 15);
 *   element i is the b-bit field at bit b*(i mod (32/b)) of word i/(32/b).
 * Code plane (MBIT): the level plane holds one m-bit code per element,
 *   uint32 [M][ld*m/32], element i in the m-bit field at bit m*(i mod (32/m))
 *   of word i/(32/m); bit m-1 of a code is the sign bit, bits 0..m-2 the
 *   level.  The sign plane is not used.
 * Scales (SIGN, QSGD, MBIT): fp32 [M][n_seg], the scale (SIGN) or sigma
 *   (QSGD, MBIT) of segment j of worker m.
 * val/idx (TOPK): fp32 and uint32 [M][k]; the selected p_i and their indices
 *   i, in ascending i, each below d.  A message that breaks this (read by
 *   dqgan_unpack or dqgan_aggregate) gives undefined values but no access
 *   outside the buffers: indices at or beyond d are skipped.
 *   dqgan_aggregate reads both lists in aligned 16-byte words: when M*k*4
 *   is not a multiple of 16, it also reads (and ignores) the bytes after the
 *   last entry up to the next 16-byte boundary, so they must be readable
 *   device memory (as in any allocation made for the buffer itself).
 *   (IDENTITY: val is the dense fp32 [M][ld] p-hat = p.)
 * Unused planes may be NULL. */
typedef struct {
    uint32_t *sign;
    uint32_t *level;
    float *scale;
    float *val;
    uint32_t *idx;
} dqgan_wire;

/* Create a plan for `desc` on the current device.  Allocates the plan's
 * device scratch (segment tables, partial norms, top-k workspace).
 * Errors: DQGAN_EINVAL for an invalid descriptor or NULL `out` (nothing is
 * allocated), DQGAN_ENOMEM, DQGAN_EHIP. */
dqgan_status dqgan_plan_create(const dqgan_desc *desc, dqgan_plan *out);

/* Free a plan and its scratch (synchronizes the plan's device first).
 * NULL is accepted and ignored. */
dqgan_status dqgan_plan_destroy(dqgan_plan plan);

/* Bytes of each message plane the caller must allocate for this plan (0 for
 * planes the compressor does not use).  Any output pointer may be NULL. */
dqgan_status dqgan_wire_bytes(dqgan_plan plan, size_t *sign, size_t *level, size_t *scale, size_t *val,
                              size_t *idx);

/* Worker side of Algorithm 2 for all M workers (EF accumulate, compress,
 * pack, EF residual): p = fl(fl(eta*g) + e); p-hat = Q(p); e <- fl(p - p-hat);
 * the message goes to `out`.
 *   G:  [M][ld] gradients g_t (read).     E: [M][ld] e_{t-1} in, e_t out.
 *   t:  iteration number (QSGD, MBIT: Philox counter word 2).
 *   scales_in: NULL to compute the segment scales from p (Section 2.4 /
 *     equation qsgd); else device fp32 [M][n_seg] scales to use instead
 *     (they are also copied to out->scale).  Ignored by TOPK and IDENTITY.
 * QSGD rounding: u = (word >> 8) * 2^-24 of Philox4x32-10 with key
 * (lo32(seed), hi32(seed)), counter (lo32(i>>2), m, t, hi32(i>>2)), output
 * word i & 3; r = fl(|p| * fl(s/sigma)), l = min(floor(r), s), level =
 * min(l + [u < r - l], s) (l = s rounds no further); p-hat =
 * copysign(fl(level * fl(sigma/s)), p); sigma = 0 gives level 0.
 * MBIT: the QSGD rule with s = k = 2^(m-1) - 1 levels.
 * SIGN: p-hat = -scale if the sign bit of p is set, else +scale.
 * TOPK: the k largest |p| (ties to the lower index); p-hat = p there, 0
 * elsewhere. */
dqgan_status dqgan_compress_ef(dqgan_plan plan, float eta, uint32_t t, const float *G, float *E,
                               const float *scales_in, const dqgan_wire *out, void *stream);

/* Pack per-element codes into the message planes (SIGN, QSGD, MBIT): the
 * worker's push of p-hat to the server in Algorithm 2, for codes the caller
 * computed itself.
 *   codes: [M][ld] uint16; bit 15 = sign bit, bits 0..14 = level (QSGD, MBIT;
 *   must be <= s, resp. k).  scales: [M][n_seg], copied to out->scale.
 * TOPK and IDENTITY return DQGAN_EUNSUPPORTED. */
dqgan_status dqgan_pack(dqgan_plan plan, const uint16_t *codes, const float *scales, const dqgan_wire *out,
                        void *stream);

/* Decode the M messages to the dense p-hat [M][ld]: what the server holds
 * after pulling the workers' pushed messages in Algorithm 2.  SIGN: +-scale; QSGD: copysign(fl(level * fl(sigma/s)),
 * sign); MBIT: the same with s = k; TOPK: val at idx, 0 elsewhere; IDENTITY:
 * val. */
dqgan_status dqgan_unpack(dqgan_plan plan, const dqgan_wire *in, float *Phat, void *stream);

/* Server average (Algorithm 2): Qhat_i = fl(S_i / M) with
 * S_i = (...((p-hat^(0)_i + p-hat^(1)_i) + p-hat^(2)_i) ... + p-hat^(M-1)_i)
 * summed in ascending worker order.  Qhat: [ld]. */
dqgan_status dqgan_aggregate(dqgan_plan plan, const dqgan_wire *in, float *Qhat, void *stream);

/* OMD update and extrapolation (Algorithm 2):
 *   W <- fl(W - Qhat)                     (w_t = w_{t-1} - q-hat_t)
 *   WX[m] = fl(W - fl(fl(eta*G[m]) + E[m])) for every m, with the updated W
 *   (w_{t+1/2}^(m) = w_t - (eta g_t^(m) + e_t^(m))).
 * E holds e_t.  WX may be NULL (update only). */
dqgan_status dqgan_omd_step(dqgan_plan plan, float eta, const float *Qhat, float *W, const float *G,
                            const float *E, float *WX, void *stream);

/* One whole iteration of Algorithm 2 (every worker step, the push of the
 * messages, the server's pull and average, the update and the next
 * evaluation points) in as few passes over HBM as the data dependences
 * allow: dqgan_compress_ef, then the server average of the M messages
 * (decoded in registers, not re-read from the message), dqgan_omd_step.
 * Results equal those of the separate calls bit for bit.
 *   G [M][ld] read; E [M][ld] e_{t-1} in, e_t out; W [ld] w_{t-1} in, w_t
 *   out; WX [M][ld] out (required); out: the message; Qhat [ld] or NULL. */
dqgan_status dqgan_step_fused(dqgan_plan plan, float eta, uint32_t t, const float *G, float *E, float *W,
                              float *WX, const dqgan_wire *out, float *Qhat, void *stream);

/* The two passes of dqgan_step_fused, for callers that schedule or time them
 * separately.  dqgan_step_scales reads G and E (e_{t-1}) once and computes
 * what the compressor must know about the whole of each worker's vector
 * before it can encode any element: the segment scales (SIGN, QSGD, MBIT;
 * written to out->scale) or the selection threshold (TOPK).  dqgan_step_apply then
 * runs the fused iteration with that state, which the plan holds in its
 * scratch: the two calls must be issued in this order on one stream with the
 * same G and E and no other call on the plan in between.  The arguments mean
 * what they mean for dqgan_step_fused; dqgan_step_scales then
 * dqgan_step_apply equals dqgan_step_fused bit for bit. */
dqgan_status dqgan_step_scales(dqgan_plan plan, float eta, const float *G, const float *E, const dqgan_wire *out,
                               void *stream);
dqgan_status dqgan_step_apply(dqgan_plan plan, float eta, uint32_t t, const float *G, float *E, float *W, float *WX,
                              const dqgan_wire *out, float *Qhat, void *stream);

/* dqgan_step_fused without a plan and without any allocation, for callers
 * that cannot allocate device memory: code under HIP graph capture, serving
 * loops and harnesses that forbid hipMalloc.  Same arguments, results and
 * buffer rules as dqgan_step_fused, with the descriptor (host; its
 * seg_offsets are read during the call) in place of the plan.
 *   Compressors: SIGN, QSGD, MBIT, IDENTITY; TOPK returns
 *   DQGAN_EUNSUPPORTED.
 *   Limit: the segment tables, the statistics pass's partial norms and the
 *   per-segment constants live in one static 8 MiB device array per device
 *   (held until the process ends).  They need about
 *   12 M P + 16 P + 8 M S + ld/256 + 12 S bytes (P = number of pieces,
 *   sum over segments of ceil(n_j / piece), piece = 32768 elements when
 *   M * floor(d / 32768) >= 16384, else 16384; S = n_seg; every table
 *   rounded up to 256 bytes); a workload above 8 MiB, or with more than 255
 *   segments, returns DQGAN_ESCRATCH and enqueues nothing.
 *   The array is shared by every call on the device and keeps the last
 *   call's contents (every table is rewritten at each call, nothing relies
 *   on earlier contents): calls that overlap on one device race.
 * Enqueues kernels only (no memset, no host synchronization). */
dqgan_status dqgan_step_fused_noalloc(const dqgan_desc *desc, float eta, uint32_t t, const float *G, float *E,
                                      float *W, float *WX, const dqgan_wire *out, float *Qhat, void *stream);

/* Static text for a status code. */
const char *dqgan_status_string(dqgan_status status);

#ifdef __cplusplus
}
#endif

#endif /* DQGAN_H */
