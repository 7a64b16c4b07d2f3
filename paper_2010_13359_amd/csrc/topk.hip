// Top-k compressor (Theorem 1 of arXiv:2010.13359: keep the k entries of
// largest magnitude; ties go to the lower index) -- the selection pass.
//
// Keys are the binary32 bit patterns of |p| (p = fl(fl(eta g) + e)), which
// order like |p|.  The selection of a row is the k largest composite keys
// (key, ~index): element i is selected iff key > T, or key == T and i <= I.
//
// Per row, with one full read of g and e:
//  1. sample: one 256-element chunk per 65536 elements, histogram of key>>16;
//  2. band: the sample ranks k/d * s -+ 8 sigma bracket the k-th key in a
//     band [lo, hi];
//  3. full pass: per 256-element tile the number of keys above hi; every
//     in-band (key, index) goes to a candidate list, each workgroup's as one
//     contiguous run (its 64 tiles), a tile that overflows its wave's
//     staging from the top of the list down;
//  4. exact radix select of the remaining rank among the candidates gives T
//     and I: the first digit of key - lo from a histogram several workgroups
//     per row build, the candidates in its bin listed, and the remaining
//     digits of key - lo (and, when the k-th key is shared and not every
//     candidate with it is taken, three digits of ~index) decided over that
//     short list by one workgroup in LDS;
//  5. selected spilled candidates are added to their tiles' counts; per
//     64-tile chunk, the selected candidates of its run are added too and
//     the tiles' offsets within the chunk are scanned; a per-row scan of the
//     chunk totals gives each chunk's first position.
// If the band missed the k-th key (or the candidates overflow the list),
// the row falls back to a full-row radix select over
// six digits of (key, ~index) (one read of the row per digit) and a recount.
// The fused apply pass then writes (value, index) in ascending index order
// from each tile's position.
#include "device.hpp"
#include "plan.hpp"

namespace dq {

namespace {

constexpr int kFbBlocks = 128;  // workgroups of the full-row search (each looping over the rows)
constexpr int kSelBlocks = 16;  // workgroups per row of a candidate histogram

__device__ __forceinline__ uint32_t key_of(float g, float e, float eta) {
    const float p = add_rn(mul_rn(eta, g), e);
    return __float_as_uint(p) & 0x7FFFFFFFu;
}

__global__ __launch_bounds__(kBlock) void k_fill_f32(float *__restrict__ p, int64_t n) {
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * kBlock)
        p[i] = 0.0f;
}

// Digit of a composite key for pass 0..5 and the filter of elements still in
// play (those whose decided digits equal the prefixes found so far).
__device__ __forceinline__ uint32_t digit_of(int pass, uint32_t key, uint32_t ni) {
    switch (pass) {
        case 0: return key >> 20;
        case 1: return (key >> 9) & 0x7FFu;
        case 2: return key & 0x1FFu;
        case 3: return ni >> 21;
        case 4: return (ni >> 10) & 0x7FFu;
        default: return ni & 0x3FFu;
    }
}
__device__ __forceinline__ bool in_play(int pass, uint32_t key, uint32_t ni, uint32_t kp, uint32_t ip) {
    switch (pass) {
        case 0: return true;
        case 1: return (key >> 20) == (kp >> 20);
        case 2: return (key >> 9) == (kp >> 9);
        case 3: return key == kp;
        case 4: return key == kp && (ni >> 21) == (ip >> 21);
        default: return key == kp && (ni >> 10) == (ip >> 10);
    }
}
__host__ __device__ __forceinline__ int bins_of(int pass) { return pass == 2 ? 512 : pass == 5 ? 1024 : 2048; }
__device__ __forceinline__ void add_prefix(int pass, uint32_t bin, uint32_t &kp, uint32_t &ip) {
    switch (pass) {
        case 0: kp |= bin << 20; break;
        case 1: kp |= bin << 9; break;
        case 2: kp |= bin; break;
        case 3: ip |= bin << 21; break;
        case 4: ip |= bin << 10; break;
        default: ip |= bin; break;
    }
}

// One wave finds, in a histogram of nb bins, the bin holding the rank-th
// largest item (rank >= 1) and the count of items in higher bins.  Returns
// false if the histogram holds fewer than rank items.
__device__ bool wave_find_desc(const uint32_t *h, int nb, uint32_t rank, uint32_t &bin, uint32_t &above) {
    // each lane holds its (at most 32) bins in registers: loaded once, in
    // parallel, and the lane that holds the rank scans them without reloads
    constexpr int kMaxPer = kDigitBins / 64;
    const int lane = threadIdx.x & 63;
    const int per = (nb + 63) / 64;
    uint32_t v[kMaxPer];
    uint32_t s = 0;
#pragma unroll
    for (int j = 0; j < kMaxPer; ++j) {
        const int b = nb - 1 - (lane * per + j);
        v[j] = (j < per && b >= 0) ? h[b] : 0u;
        s += v[j];
    }
    uint32_t incl = s;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t x = __shfl_up(incl, o);
        if (lane >= o) incl += x;
    }
    const uint32_t excl = incl - s;
    const uint64_t hit = __ballot(excl < rank && rank <= incl);
    if (!hit) return false;
    const int L = __ffsll(static_cast<unsigned long long>(hit)) - 1;
    uint32_t rb = 0, ra = 0;
    if (lane == L) {
        uint32_t acc = excl;
        bool found = false;
#pragma unroll
        for (int j = 0; j < kMaxPer; ++j) {
            const int b = nb - 1 - (lane * per + j);
            if (!found && j < per && b >= 0 && acc + v[j] >= rank) {
                rb = static_cast<uint32_t>(b);
                ra = acc;
                found = true;
            }
            acc += found ? 0u : v[j];
        }
    }
    bin = __shfl(rb, L);
    above = __shfl(ra, L);
    return true;
}

// 1. Sample histogram of key >> 16 (one 256-element chunk per 65536 elements).
// The 128 KiB LDS histogram allows one workgroup per CU, so a row has few
// workgroups (each flushes its nonzero bins with global atomics) and each
// of their 16 waves keeps four chunks' loads in flight.
constexpr int kSampleThreads = 1024;
constexpr int kSampleBlocks = 4;  // workgroups per row
constexpr int kSampleU = 4;       // chunks in flight per wave

__global__ __launch_bounds__(kSampleThreads) void k_topk_sample(const float *__restrict__ G,
                                                                const float *__restrict__ E, float eta, int64_t d,
                                                                int64_t ld, int64_t n_chunks,
                                                                uint32_t *__restrict__ hist) {
    constexpr int kWaves = kSampleThreads / 64;
    __shared__ uint32_t h[kSampleBins];
    const int m = blockIdx.y;
    for (int b = threadIdx.x; b < kSampleBins; b += kSampleThreads) h[b] = 0;
    __syncthreads();
    const float *g = G + static_cast<int64_t>(m) * ld;
    const float *e = E + static_cast<int64_t>(m) * ld;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kWaves;
    for (int64_t c0 = static_cast<int64_t>(blockIdx.x) * kWaves + wave; c0 < n_chunks; c0 += stride * kSampleU) {
        f32x4 gv[kSampleU], ev[kSampleU];
#pragma unroll
        for (int u = 0; u < kSampleU; ++u) {
            // chunks past the row's last are not examined; their loads read
            // the first chunk (always in bounds)
            const int64_t c = c0 + stride * u;
            const int64_t i0 = (c < n_chunks ? c * kSampleStride : 0) + 4 * lane;
            gv[u] = ld4(g + i0);
            ev[u] = ld4(e + i0);
        }
#pragma unroll
        for (int u = 0; u < kSampleU; ++u) {
            const int64_t c = c0 + stride * u;
            const int64_t i0 = c * kSampleStride + 4 * lane;
            if (c < n_chunks && i0 < d) {
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    if (i0 + k < d) atomicAdd(&h[key_of(elem(gv[u], k), elem(ev[u], k), eta) >> 16], 1u);
            }
        }
    }
    __syncthreads();
    uint32_t *hm = hist + static_cast<int64_t>(m) * kSampleBins;
    for (int b = threadIdx.x; b < kSampleBins; b += kSampleThreads)
        if (h[b]) atomicAdd(&hm[b], h[b]);
}

// Exclusive prefix sum of v over the 1024 threads of a workgroup (wsum: 16
// words of LDS); total receives the sum over all threads.
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t *wsum, uint32_t &total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t incl = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t x = __shfl_up(incl, o);
        if (lane >= o) incl += x;
    }
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    uint32_t wbase = 0, tot = 0;
    for (int w = 0; w < 16; ++w) {
        if (w < wave) wbase += wsum[w];
        tot += wsum[w];
    }
    total = tot;
    return wbase + incl - v;
}

// 2. Band: the sample ranks k/d * s -+ 8 sigma (binomial) bracket the k-th
// key; the bins where the count from the top reaches them bound [lo, hi].
__global__ __launch_bounds__(1024) void k_topk_band(uint32_t *__restrict__ hist, uint32_t *__restrict__ sel_hist,
                                                    TopkRow *__restrict__ rows, uint32_t *__restrict__ ctr,
                                                    uint32_t n_samples, int64_t d, int64_t k) {
    // thread t holds the t-th group of kPer bins counted from the top; a
    // block scan finds the group where the count from the top reaches a
    // rank, and that thread finds the bin in its registers.
    constexpr int kPer = kSampleBins / 1024;
    __shared__ uint32_t wsum[16];
    __shared__ uint32_t found[2];
    const int m = blockIdx.x;
    const int t = threadIdx.x;
    const uint32_t *h = hist + static_cast<int64_t>(m) * kSampleBins;
    uint32_t asc[kPer];  // bins kSampleBins - kPer (t+1) .. kSampleBins - kPer t - 1, ascending
    const uint4 *src = reinterpret_cast<const uint4 *>(h + kSampleBins - kPer * (t + 1));
#pragma unroll
    for (int q = 0; q < kPer / 4; ++q) {
        const uint4 v = src[q];
        asc[4 * q] = v.x;
        asc[4 * q + 1] = v.y;
        asc[4 * q + 2] = v.z;
        asc[4 * q + 3] = v.w;
    }
    // the histogram is zeroed once read (the next iteration's sample starts
    // from zero), and so are the row's candidate digit histograms
    uint4 *dst = reinterpret_cast<uint4 *>(hist + static_cast<int64_t>(m) * kSampleBins + kSampleBins - kPer * (t + 1));
#pragma unroll
    for (int q = 0; q < kPer / 4; ++q) dst[q] = make_uint4(0u, 0u, 0u, 0u);
    for (int b = t; b < kDigitBins; b += 1024) sel_hist[static_cast<int64_t>(m) * kDigitBins + b] = 0u;
    uint32_t s = 0;
#pragma unroll
    for (int j = 0; j < kPer; ++j) s += asc[j];
    if (t == 0) found[0] = found[1] = 0xFFFFFFFFu;
    uint32_t total;
    const uint32_t excl = block_exclusive_scan(s, wsum, total);  // count above this group
    const double f = static_cast<double>(k) / static_cast<double>(d);
    const double ns = static_cast<double>(n_samples);
    const double mean = f * ns;
    const double sd = sqrt(ns * f * (1.0 - f)) + 1.0;
    const double z = 8.0;
    const double a = floor(mean - z * sd);
    const double c = ceil(mean + z * sd);
    // ranks (from the top) whose bins bound the band: a + 1 for hi, c for lo
    const uint32_t want[2] = {a >= 1.0 ? static_cast<uint32_t>(a) + 1u : 0u,
                              c <= ns ? static_cast<uint32_t>(c) : 0u};
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        const uint32_t rank = want[r];
        if (rank != 0u && excl < rank && rank <= excl + s) {
            uint32_t acc = excl;
            for (int j = 0; j < kPer; ++j) {
                const uint32_t cnt = asc[kPer - 1 - j];
                if (acc + cnt >= rank) {
                    found[r] = static_cast<uint32_t>(kSampleBins - 1 - (kPer * t + j));
                    break;
                }
                acc += cnt;
            }
        }
    }
    __syncthreads();
    if (t == 0) {
        uint32_t hi = 0x7FFFFFFFu, lo = 0u;
        if (found[0] != 0xFFFFFFFFu) hi = ((found[0] + 1u) << 16) - 1u;
        if (found[1] != 0xFFFFFFFFu) lo = found[1] << 16;
        if (lo > hi) lo = 0u;
        TopkRow row{};
        row.lo = lo;
        row.hi = hi;
        rows[m] = row;
        uint32_t *c = ctr + static_cast<int64_t>(m) * kRowCtrWords;
        c[kCtrCand] = c[kCtrAbove] = c[kCtrSpill] = c[kCtrPlay] = 0u;
    }
}

// 3. Full pass: per tile the count of keys above the band, and the in-band
// candidates appended to the row's list.  A workgroup covers 64 consecutive
// tiles of one row; wave w owns 16 consecutive tiles of them, four per round
// (the round's eight loads issued before its first tile is examined).  Lane j
// of a wave keeps the count of the wave's j-th tile, and the wave writes its
// 16 counts (16-bit) with one 32-byte store at the end: over 64 rows of
// 10^8 elements a 4-byte count store per tile held the pass 8 % above its
// loads alone.
// Candidates are staged in the wave's quarter of an LDS buffer with a
// wave-uniform count; at the end the workgroup adds its above-band total
// (the sum of its tile counts) to the row's counters and writes its
// candidates as one run from the bottom of the row's list, whose place it
// records for the per-chunk count.  A tile whose
// candidates do not fit the wave's quarter (more than 256 in-band keys in
// its 4096 elements: a segment whose scale puts most of it in the band)
// stores them from the top of the list down ("spills").  A tile wholly below d
// (all but the last of a row) is classified without per-element bounds
// tests, on masks taken straight from the comparisons.
constexpr int kPassRounds = 4;
constexpr int kPassTilesPerWave = 4 * kPassRounds;
constexpr int kPassTilesPerBlock = kPassTilesPerWave * (kBlock / 64);
__global__ __launch_bounds__(kBlock) void k_topk_pass(const float *__restrict__ G, const float *__restrict__ E,
                                                      float eta, int64_t d, int64_t ld, int64_t n_tiles,
                                                      const TopkRow *__restrict__ rows, uint32_t *__restrict__ ctr,
                                                      uint16_t *__restrict__ tile_cnt, uint32_t *__restrict__ ckey,
                                                      uint32_t *__restrict__ cidx,
                                                      int64_t cap, uint2 *__restrict__ runs, int64_t n_chunks) {
    constexpr uint32_t kStage = 256;  // staged candidates per wave
    constexpr int kWaves = kBlock / 64;
    __shared__ uint2 buf[kWaves][kStage];
    __shared__ uint32_t wave_nab[kWaves], wave_ns[kWaves], base;
    const int m = blockIdx.y;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t lo = rows[m].lo, hi = rows[m].hi;
    const float *g = G + static_cast<int64_t>(m) * ld;
    const float *e = E + static_cast<int64_t>(m) * ld;
    const uint32_t span = hi - lo;
    uint32_t *krow = ckey + static_cast<int64_t>(m) * cap;
    uint32_t *irow = cidx + static_cast<int64_t>(m) * cap;
    uint2 *stage = buf[wave];
    const int64_t t0 = static_cast<int64_t>(blockIdx.x) * kPassTilesPerBlock + kPassTilesPerWave * wave;
    uint32_t my_cnt = 0;  // lane j < 16: above-band count of tile t0 + j
    uint32_t ns = 0;      // wave-uniform: candidates staged by the wave
    for (int round = 0; round < kPassRounds; ++round) {
        // Unconditional loads (a tile past the row's end reads the last tile
        // again and is not examined): loads under a branch made the compiler
        // wait for each tile's loads before issuing the next tile's.
        f32x4 gvs[4], evs[4];
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            const int64_t tile = t0 + 4 * round + it;
            const int64_t i0 = (tile < n_tiles ? tile : n_tiles - 1) * kTopkTile + 4 * lane;
            gvs[it] = ld_stream(g + i0);
            evs[it] = ld_stream(e + i0);
        }
#pragma unroll
        for (int it = 0; it < 4; ++it) {
            // A tile past the row's end (only in a row's last workgroup) is
            // examined too, with no element valid; the loads stay ahead of
            // every tile's work only if no tile's work is conditional.
            const int64_t tile = t0 + 4 * round + it;
            const int64_t i0 = tile * kTopkTile + 4 * lane;
            const int64_t end = tile < n_tiles ? d : 0;  // elements [0, end) of the row are valid here
            // Only the last tile of a row can hold elements at or beyond d.
            const bool full = (tile + 1) * kTopkTile <= end;
            uint32_t keys[4];
            uint64_t cb[4];  // wave masks of the in-band candidates, per element of the quad
            uint32_t above_n = 0, tot = 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) keys[k] = key_of(elem(gvs[it], k), elem(evs[it], k), eta);
            if (full) {
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    above_n += __popcll(__builtin_amdgcn_ballot_w64(keys[k] > hi));
                    cb[k] = __builtin_amdgcn_ballot_w64(keys[k] - lo <= span);  // lo <= key <= hi
                    tot += __popcll(cb[k]);
                }
            } else {
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const bool valid = i0 + k < end;
                    above_n += __popcll(__builtin_amdgcn_ballot_w64(valid && keys[k] > hi));
                    cb[k] = __builtin_amdgcn_ballot_w64(valid && keys[k] - lo <= span);
                    tot += __popcll(cb[k]);
                }
            }
            my_cnt = lane == 4 * round + it ? above_n : my_cnt;
            if (tot) {
                // this lane's first slot: the wave's candidates in lower lanes
                uint32_t pre = 0;
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    pre = __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(cb[k] >> 32),
                                                    __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(cb[k]), pre));
                if (ns + tot <= kStage) {
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        if ((cb[k] >> lane) & 1u) {
                            stage[ns + pre] = make_uint2(keys[k], static_cast<uint32_t>(i0 + k));
                            ++pre;
                        }
                    }
                    ns += tot;
                } else {
                    // the wave's staging is full: these go to the top of the
                    // row's list, counted per tile by k_topk_spill_count
                    uint32_t sbase = 0;
                    if (lane == 0) sbase = atomicAdd(ctr + static_cast<int64_t>(m) * kRowCtrWords + kCtrSpill, tot);
                    sbase = __builtin_amdgcn_readfirstlane(sbase);
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        if ((cb[k] >> lane) & 1u) {
                            const int64_t j = static_cast<int64_t>(sbase) + pre;
                            if (j < cap) {
                                krow[cap - 1 - j] = keys[k];
                                irow[cap - 1 - j] = static_cast<uint32_t>(i0 + k);
                            }
                            ++pre;
                        }
                    }
                }
            }
        }
    }
    // the wave's 16 tile counts: lanes 0..15, one contiguous store
    if (lane < kPassTilesPerWave && t0 + lane < n_tiles)
        tile_cnt[static_cast<int64_t>(m) * n_tiles + t0 + lane] = static_cast<uint16_t>(my_cnt);
    // keys above the band in the wave's tiles: the sum of its 16 tile counts
    uint32_t nab = my_cnt;
#pragma unroll
    for (int o = 1; o < kPassTilesPerWave; o <<= 1) nab += __shfl_xor(nab, o);
    if (lane == 0) {
        wave_nab[wave] = nab;
        wave_ns[wave] = ns;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t a = 0, n = 0;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            a += wave_nab[w];
            n += wave_ns[w];
        }
        uint32_t *c = ctr + static_cast<int64_t>(m) * kRowCtrWords;
        if (a) atomicAdd(c + kCtrAbove, a);
        base = n ? atomicAdd(c + kCtrCand, n) : 0u;
        runs[static_cast<int64_t>(m) * n_chunks + blockIdx.x] = make_uint2(base, n);
    }
    __syncthreads();
    uint32_t off = base;
    for (int w = 0; w < wave; ++w) off += wave_ns[w];
    for (uint32_t j = lane; j < ns; j += 64) {
        const int64_t pos = static_cast<int64_t>(off) + j;
        if (pos < cap) {
            const uint2 c = stage[j];
            krow[pos] = c.x;
            irow[pos] = c.y;
        }
    }
}

// 4. Exact selection among the candidates.  A row's search is on when its
// candidates hold the k-th key: all staged, within the list, and the keys
// above the band fewer than k with the rest of k among the candidates.
__device__ __forceinline__ uint64_t n_listed(const TopkRow &r) {
    return static_cast<uint64_t>(r.n_cand) + r.n_spill;
}
__device__ __forceinline__ bool sel_ok(const TopkRow &r, int64_t k, int64_t cap) {
    return n_listed(r) <= static_cast<uint64_t>(cap) && r.n_above < static_cast<uint64_t>(k) &&
           static_cast<uint64_t>(k) - r.n_above <= n_listed(r);
}
// The place of candidate j in a row's list: the runs [0, n_cand), then the
// spills stored from the top down.  The list is two planes of the row's
// capacity, keys and indices, so that a search that needs only the keys
// reads half the bytes.
// Inclusive prefix sum over the 64 lanes of a wave, all of them active, by
// data-parallel-primitive moves: shifts by 1, 2, 4 and 8 lanes inside each
// row of 16 lanes (a lane whose source lies before its row reads 0), then
// the last lane of rows 0 and 2 added to rows 1 and 3, then the last lane of
// row 1 added to rows 2 and 3.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
    x += __builtin_amdgcn_update_dpp(0u, x, 0x111, 0xF, 0xF, true);   // row_shr:1
    x += __builtin_amdgcn_update_dpp(0u, x, 0x112, 0xF, 0xF, true);   // row_shr:2
    x += __builtin_amdgcn_update_dpp(0u, x, 0x114, 0xF, 0xF, true);   // row_shr:4
    x += __builtin_amdgcn_update_dpp(0u, x, 0x118, 0xF, 0xF, true);   // row_shr:8
    x += __builtin_amdgcn_update_dpp(0u, x, 0x142, 0xA, 0xF, false);  // row_bcast:15, rows 1 and 3
    x += __builtin_amdgcn_update_dpp(0u, x, 0x143, 0xC, 0xF, false);  // row_bcast:31, rows 2 and 3
    return x;
}

__device__ __forceinline__ uint64_t cand_pos(uint64_t j, uint32_t n_cand, int64_t cap) {
    return j < n_cand ? j : static_cast<uint64_t>(cap) - 1 - (j - n_cand);
}

// The search over the candidates: the first digit of key - lo (its top 11
// bits, or all of them when narrower) from a histogram that kSelBlocks
// workgroups per row build over the whole list; the candidates in that
// digit's bin -- a few hundred or thousand in a typical row -- are then
// listed once, and one workgroup per row decides the remaining digits of
// key - lo and, when the k-th key is shared and not every candidate with it
// is taken, three digits of ~index, all in LDS over that list.
struct TopState {
    uint32_t rank;   // rank still to place among the candidates in play
    uint32_t kp;     // decided high bits of key - lo
    int top;         // bits of key - lo not yet decided
};

__device__ __forceinline__ int key_width(const TopkRow &r) {
    const uint32_t span = r.hi - r.lo;
    int width = 0;
    while (width < 32 && (span >> width) != 0u) ++width;  // bits of key - lo
    return width;
}

// The state after the first digit (one wave replays it from the histogram).
__device__ TopState sel_first_digit(const TopkRow &r, int64_t k, const uint32_t *__restrict__ h) {
    TopState s;
    s.rank = static_cast<uint32_t>(static_cast<uint64_t>(k) - r.n_above);
    s.kp = 0u;
    s.top = key_width(r);
    if (s.top > 0) {
        const int wbits = s.top < 11 ? s.top : 11;
        const int shift = s.top - wbits;
        uint32_t bin = 0, above = 0;
        wave_find_desc(h, 1 << wbits, s.rank, bin, above);
        s.rank -= above;
        s.kp = bin << shift;
        s.top = shift;
    }
    return s;
}

constexpr int kSelU = 8;  // candidates in flight per thread

// The first key digit's histogram (kSelBlocks workgroups per row).
__global__ __launch_bounds__(kBlock) void k_topk_sel_top(TopkRow *__restrict__ rows, const uint32_t *__restrict__ ctr,
                                                         const uint32_t *__restrict__ ckey, int64_t cap, int64_t k,
                                                         uint32_t *__restrict__ sel_hist) {
    __shared__ uint32_t h[kDigitBins];
    const int m = blockIdx.y;
    TopkRow r = rows[m];
    const uint32_t *c = ctr + static_cast<int64_t>(m) * kRowCtrWords;
    r.n_cand = c[kCtrCand];
    r.n_above = c[kCtrAbove];
    r.n_spill = c[kCtrSpill];
    // the later kernels read the counters from the row record (the other
    // workgroups of this launch may read the record meanwhile: they take
    // the counters from ctr, and the rest of the record does not change)
    if (blockIdx.x == 0 && threadIdx.x == 0) {
        rows[m].n_cand = r.n_cand;
        rows[m].n_above = r.n_above;
        rows[m].n_spill = r.n_spill;
    }
    const int width = key_width(r);
    if (!sel_ok(r, k, cap) || width == 0) return;
    const int wbits = width < 11 ? width : 11;
    const int shift = width - wbits;
    const int nb = 1 << wbits;
    for (int b = threadIdx.x; b < nb; b += kBlock) h[b] = 0u;
    __syncthreads();
    const uint32_t *krow = ckey + static_cast<int64_t>(m) * cap;
    const uint64_t n = n_listed(r);
    const uint64_t per = (n + kSelBlocks - 1) / kSelBlocks;
    const uint64_t j_lo = per * blockIdx.x, j_hi = j_lo + per < n ? j_lo + per : n;
    for (uint64_t j0 = j_lo + threadIdx.x; j0 < j_hi; j0 += static_cast<uint64_t>(kBlock) * kSelU) {
        uint32_t keys[kSelU];
#pragma unroll
        for (int u = 0; u < kSelU; ++u) {
            const uint64_t j = j0 + static_cast<uint64_t>(kBlock) * u;
            keys[u] = j < j_hi ? krow[cand_pos(j, r.n_cand, cap)] : 0u;
        }
#pragma unroll
        for (int u = 0; u < kSelU; ++u)
            if (j0 + static_cast<uint64_t>(kBlock) * u < j_hi) atomicAdd(&h[(keys[u] - r.lo) >> shift], 1u);
    }
    __syncthreads();
    uint32_t *hm = sel_hist + static_cast<int64_t>(m) * kDigitBins;
    for (int b = threadIdx.x; b < nb; b += kBlock)
        if (h[b]) atomicAdd(&hm[b], h[b]);
}

// The candidates in the first digit's bin, listed (kSelBlocks workgroups per
// row; one atomic per wave and round).
__global__ __launch_bounds__(kBlock) void k_topk_sel_collect(const TopkRow *__restrict__ rows,
                                                             uint32_t *__restrict__ ctr,
                                                             const uint32_t *__restrict__ ckey,
                                                             const uint32_t *__restrict__ cidx, int64_t cap, int64_t k,
                                                             const uint32_t *__restrict__ sel_hist,
                                                             uint2 *__restrict__ play) {
    __shared__ TopState st;
    const int m = blockIdx.y;
    const TopkRow r = rows[m];
    if (!sel_ok(r, k, cap)) return;
    if (threadIdx.x < 64) {
        const TopState s = sel_first_digit(r, k, sel_hist + static_cast<int64_t>(m) * kDigitBins);
        if (threadIdx.x == 0) st = s;
    }
    __syncthreads();
    const TopState s = st;
    const int lane = threadIdx.x & 63;
    const uint32_t *krow = ckey + static_cast<int64_t>(m) * cap;
    const uint32_t *irow = cidx + static_cast<int64_t>(m) * cap;
    uint2 *prow = play + static_cast<int64_t>(m) * cap;
    const uint64_t n = n_listed(r);
    const uint64_t per = (n + kSelBlocks - 1) / kSelBlocks;
    const uint64_t j_lo = per * blockIdx.x, j_hi = j_lo + per < n ? j_lo + per : n;
    // rounds of kSelU * kBlock candidates (all loaded before the first is
    // examined; every thread of the workgroup in each round), one atomic per
    // wave and round
    for (uint64_t jb = j_lo; jb < j_hi; jb += static_cast<uint64_t>(kBlock) * kSelU) {
        uint32_t ks[kSelU];  // keys; a candidate's index is read only when it is listed
        uint64_t mask[kSelU];
        uint32_t tot = 0;
#pragma unroll
        for (int u = 0; u < kSelU; ++u) {
            const uint64_t j = jb + static_cast<uint64_t>(kBlock) * u + threadIdx.x;
            ks[u] = j < j_hi ? krow[cand_pos(j, r.n_cand, cap)] : 0u;
        }
#pragma unroll
        for (int u = 0; u < kSelU; ++u) {
            const uint64_t j = jb + static_cast<uint64_t>(kBlock) * u + threadIdx.x;
            const uint32_t rel = ks[u] - r.lo;
            mask[u] = __ballot(j < j_hi && (s.top >= 32 || (rel >> s.top) == (s.kp >> s.top)));
            tot += __popcll(mask[u]);
        }
        if (tot) {
            uint32_t base = 0;
            if (lane == 0) base = atomicAdd(ctr + static_cast<int64_t>(m) * kRowCtrWords + kCtrPlay, tot);
            base = __builtin_amdgcn_readfirstlane(base);
#pragma unroll
            for (int u = 0; u < kSelU; ++u) {
                if ((mask[u] >> lane) & 1u) {
                    const uint32_t at = base + __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask[u] >> 32),
                                                                         __builtin_amdgcn_mbcnt_lo(
                                                                             static_cast<uint32_t>(mask[u]), 0u));
                    const uint64_t j = jb + static_cast<uint64_t>(kBlock) * u + threadIdx.x;
                    if (at < cap) prow[at] = make_uint2(ks[u], irow[cand_pos(j, r.n_cand, cap)]);
                }
                base += static_cast<uint32_t>(__popcll(mask[u]));
            }
        }
    }
}

// The search's result (one workgroup per row): the remaining digits of
// key - lo and, if needed, of ~index over the listed candidates; or the
// hand-over of the row to the full-row search (whose digit histograms are
// zeroed here).
__device__ __forceinline__ void block_find(const uint32_t *h, int nb, uint32_t rank, uint32_t *res) {
    if (threadIdx.x < 64) {
        uint32_t bin = 0, above = 0;
        wave_find_desc(h, nb, rank, bin, above);
        if (threadIdx.x == 0) {
            res[0] = bin;
            res[1] = above;
            res[2] = h[bin];
        }
    }
    __syncthreads();
}

__global__ __launch_bounds__(1024) void k_topk_sel_finish(TopkRow *__restrict__ rows, const uint32_t *__restrict__ ctr,
                                                          int64_t cap, int64_t k,
                                                          const uint32_t *__restrict__ sel_hist,
                                                          const uint2 *__restrict__ play,
                                                          uint32_t *__restrict__ fb_hist) {
    __shared__ uint32_t h[kDigitBins];
    __shared__ TopState st;
    __shared__ uint32_t res[3];
    const int m = blockIdx.x;
    const TopkRow r = rows[m];
    if (!sel_ok(r, k, cap)) {
        uint32_t *f6 = fb_hist + static_cast<int64_t>(m) * kSelectPasses * kDigitBins;
        for (int b = threadIdx.x; b < kSelectPasses * kDigitBins; b += 1024) f6[b] = 0u;
        if (threadIdx.x == 0) rows[m].fallback = 1u;
        return;
    }
    if (threadIdx.x < 64) {
        const TopState s = sel_first_digit(r, k, sel_hist + static_cast<int64_t>(m) * kDigitBins);
        if (threadIdx.x == 0) st = s;
    }
    __syncthreads();
    uint32_t rank = st.rank, kp = st.kp;
    int top = st.top;
    const uint2 *prow = play + static_cast<int64_t>(m) * cap;
    const uint32_t n_play = ctr[static_cast<int64_t>(m) * kRowCtrWords + kCtrPlay];
    const uint32_t n = n_play < cap ? n_play : static_cast<uint32_t>(cap);
    uint32_t n_bin = n;
    // remaining digits of key - lo
    while (top > 0) {
        const int wbits = top < 11 ? top : 11;
        const int shift = top - wbits;
        const int nb = 1 << wbits;
        for (int b = threadIdx.x; b < nb; b += 1024) h[b] = 0u;
        __syncthreads();
        for (uint32_t j = threadIdx.x; j < n; j += 1024) {
            const uint32_t rel = prow[j].x - r.lo;
            if (top >= 32 || (rel >> top) == (kp >> top)) atomicAdd(&h[(rel >> shift) & (nb - 1)], 1u);
        }
        __syncthreads();
        block_find(h, nb, rank, res);
        rank -= res[1];
        kp |= res[0] << shift;
        n_bin = res[2];
        top = shift;
        __syncthreads();
    }
    const uint32_t T = r.lo + kp;
    uint32_t I = 0xFFFFFFFFu;
    if (rank != n_bin) {
        // the k-th key is shared and not all of its candidates are taken:
        // three digits of ~index among them (smaller index first)
        uint32_t ip = 0u;
        for (int pass = 3; pass < 6; ++pass) {
            const int nb = bins_of(pass);
            for (int b = threadIdx.x; b < nb; b += 1024) h[b] = 0u;
            __syncthreads();
            for (uint32_t j = threadIdx.x; j < n; j += 1024) {
                const uint2 c = prow[j];
                const uint32_t ni = ~c.y;
                if (in_play(pass, c.x, ni, T, ip)) atomicAdd(&h[digit_of(pass, c.x, ni)], 1u);
            }
            __syncthreads();
            block_find(h, nb, rank, res);
            uint32_t kd = 0;
            rank -= res[1];
            add_prefix(pass, res[0], kd, ip);
            __syncthreads();
        }
        I = ~ip;
    }
    if (threadIdx.x == 0) {
        rows[m].T = T;
        rows[m].I = I;
    }
}

// 6. Full-row search of a row whose band missed: six digits of (key, ~index)
// over the whole row, one histogram slot per digit.  The kernels loop over
// the rows (a 1-D grid of kFbBlocks workgroups), so that when no row falls
// back -- the usual case -- each launch is a short loop over the row flags.
constexpr int kMaxRows = 1024;  // the library's largest worker count

// The rows that fell back, gathered into LDS by the whole workgroup with one
// parallel read of the flags (the order does not matter: rows are
// independent).  Returns their number.
__device__ int gather_fallback_rows(const TopkRow *__restrict__ rows, int M, int *fb_rows, int *n_fb) {
    if (threadIdx.x == 0) *n_fb = 0;
    __syncthreads();
    for (int m = threadIdx.x; m < M; m += kBlock)
        if (rows[m].fallback) fb_rows[atomicAdd(n_fb, 1)] = m;
    __syncthreads();
    return *n_fb;
}

struct FbState {
    uint32_t rank, kprefix, iprefix, T, I;
    int next;  // the digit whose histogram comes next, or kSelectPasses when decided
};

__device__ FbState fb_replay(int64_t k, const uint32_t *__restrict__ f6, int upto) {
    FbState s{static_cast<uint32_t>(k), 0u, 0u, 0u, 0xFFFFFFFFu, 0};
    for (int pass = 0; pass < kSelectPasses; ++pass) {
        if (pass >= upto) {
            s.next = pass;
            return s;
        }
        uint32_t bin = 0, above = 0;
        wave_find_desc(f6 + pass * kDigitBins, bins_of(pass), s.rank, bin, above);
        const uint32_t n_bin = f6[pass * kDigitBins + bin];
        s.rank -= above;
        add_prefix(pass, bin, s.kprefix, s.iprefix);
        if (pass == 2) {
            s.T = s.kprefix;
            if (s.rank == n_bin) {  // every element with key T is taken
                s.next = kSelectPasses;
                return s;
            }
        }
        if (pass == 5) s.I = ~s.iprefix;
    }
    s.next = kSelectPasses;
    return s;
}

__global__ __launch_bounds__(kBlock) void k_topk_fb_hist(int pass, const float *__restrict__ G,
                                                         const float *__restrict__ E, float eta, int64_t d, int64_t ld,
                                                         int32_t M, int64_t k, const TopkRow *__restrict__ rows,
                                                         uint32_t *__restrict__ fb_hist) {
    __shared__ uint32_t h[kDigitBins];
    __shared__ FbState st;
    __shared__ int fb_rows[kMaxRows];
    __shared__ int n_fb;
    const int nf = gather_fallback_rows(rows, M, fb_rows, &n_fb);
    for (int q = 0; q < nf; ++q) {
        const int m = fb_rows[q];
        uint32_t *f6 = fb_hist + static_cast<int64_t>(m) * kSelectPasses * kDigitBins;
        if (threadIdx.x < 64) {
            const FbState s = fb_replay(k, f6, pass);
            if (threadIdx.x == 0) st = s;
        }
        __syncthreads();
        const FbState s = st;
        if (s.next == pass) {
            const int nb = bins_of(pass);
            for (int b = threadIdx.x; b < nb; b += kBlock) h[b] = 0u;
            __syncthreads();
            const float *g = G + static_cast<int64_t>(m) * ld;
            const float *e = E + static_cast<int64_t>(m) * ld;
            const int64_t nq = (d + 3) / 4;
            for (int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; q < nq;
                 q += static_cast<int64_t>(gridDim.x) * kBlock) {
                const f32x4 gv = ld4(g + 4 * q), ev = ld4(e + 4 * q);
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int64_t i = 4 * q + c;
                    if (i < d) {
                        const uint32_t key = key_of(elem(gv, c), elem(ev, c), eta);
                        const uint32_t ni = ~static_cast<uint32_t>(i);
                        if (in_play(pass, key, ni, s.kprefix, s.iprefix)) atomicAdd(&h[digit_of(pass, key, ni)], 1u);
                    }
                }
            }
            __syncthreads();
            for (int b = threadIdx.x; b < nb; b += kBlock)
                if (h[b]) atomicAdd(&f6[pass * kDigitBins + b], h[b]);
        }
        __syncthreads();  // st and h are reused for the next row
    }
}

// ... then the selection of each fallen-back row per tile (and T, I).
__global__ __launch_bounds__(kBlock) void k_topk_fb_recount(const float *__restrict__ G, const float *__restrict__ E,
                                                            float eta, int64_t d, int64_t ld, int64_t n_tiles,
                                                            int32_t M, int64_t k, TopkRow *__restrict__ rows,
                                                            const uint32_t *__restrict__ fb_hist,
                                                            uint16_t *__restrict__ tile_cnt) {
    __shared__ FbState st;
    __shared__ int fb_rows[kMaxRows];
    __shared__ int n_fb;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nf = gather_fallback_rows(rows, M, fb_rows, &n_fb);
    for (int q = 0; q < nf; ++q) {
        const int m = fb_rows[q];
        if (threadIdx.x < 64) {
            const FbState s = fb_replay(k, fb_hist + static_cast<int64_t>(m) * kSelectPasses * kDigitBins,
                                        kSelectPasses);
            if (threadIdx.x == 0) st = s;
        }
        __syncthreads();
        const FbState s = st;
        if (blockIdx.x == 0 && threadIdx.x == 0) {
            rows[m].T = s.T;
            rows[m].I = s.I;
        }
        const float *g = G + static_cast<int64_t>(m) * ld;
        const float *e = E + static_cast<int64_t>(m) * ld;
        for (int64_t tile = static_cast<int64_t>(blockIdx.x) * 4 + wave; tile < n_tiles;
             tile += static_cast<int64_t>(gridDim.x) * 4) {
            const int64_t i0 = tile * kTopkTile + 4 * lane;
            const f32x4 gv = ld4(g + i0), ev = ld4(e + i0);
            uint32_t n = 0;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const int64_t i = i0 + c;
                const uint32_t key = key_of(elem(gv, c), elem(ev, c), eta);
                const bool sel = i < d && (key > s.T || (key == s.T && static_cast<uint32_t>(i) <= s.I));
                n += __popcll(__ballot(sel));
            }
            if (lane == 0) tile_cnt[static_cast<int64_t>(m) * n_tiles + tile] = static_cast<uint16_t>(n);
        }
        __syncthreads();  // st is reused for the next row
    }
}

// Spilled candidates (stored from the top of the list) added to their tiles'
// counts, for rows whose candidate search decided; nothing to do for most
// rows (a short exit).
constexpr int kSpillBlocks = 16;  // workgroups per row

__global__ __launch_bounds__(kBlock) void k_topk_spill_count(const TopkRow *__restrict__ rows,
                                                             const uint32_t *__restrict__ ckey,
                                                             const uint32_t *__restrict__ cidx, int64_t cap,
                                                             uint16_t *__restrict__ tile_cnt, int64_t n_tiles) {
    const int m = blockIdx.y;
    const TopkRow r = rows[m];
    if (r.fallback || r.n_spill == 0) return;
    const uint32_t *krow = ckey + static_cast<int64_t>(m) * cap;
    const uint32_t *irow = cidx + static_cast<int64_t>(m) * cap;
    // 32-bit atomics on the word holding the tile's 16-bit count (n_tiles is
    // a multiple of 4, so a row's counts start on a word; a count stays at
    // most 256 and never carries into its neighbour)
    uint32_t *trow = reinterpret_cast<uint32_t *>(tile_cnt + static_cast<int64_t>(m) * n_tiles);
    const int64_t n = r.n_spill;  // at most cap - n_cand (the search decided)
    for (int64_t j = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; j < n;
         j += static_cast<int64_t>(gridDim.x) * kBlock) {
        const uint2 c = make_uint2(krow[cap - 1 - j], irow[cap - 1 - j]);
        if (c.x > r.T || (c.x == r.T && c.y <= r.I)) {
            const uint32_t tile = c.y / kTopkTile;
            atomicAdd(&trow[tile >> 1], 1u << (16u * (tile & 1u)));
        }
    }
}

// 7. Per chunk of kTopkChunkTiles tiles: the selected candidates of the
// chunk's run added to its tiles' counts, the tiles' offsets within the
// chunk (exclusive scan) and the chunk's total.  A wave takes
// kScanChunksPerWave consecutive chunks, their counts and runs loaded before
// the first is examined (one chunk per wave made the launch a hundred
// thousand tiny workgroups).  A fallen-back row's counts come whole from the
// recount.
constexpr int kScanChunksPerWave = 4;

__global__ __launch_bounds__(kBlock) void k_topk_count_scan(const TopkRow *__restrict__ rows,
                                                            const uint32_t *__restrict__ ckey,
                                                            const uint32_t *__restrict__ cidx, int64_t cap,
                                                            const uint2 *__restrict__ runs,
                                                            const uint16_t *__restrict__ tile_cnt,
                                                            uint16_t *__restrict__ tile_off,
                                                            uint32_t *__restrict__ chunk_sum, int64_t n_tiles,
                                                            int64_t n_chunks) {
    __shared__ uint32_t sel_all[kBlock / 64][kTopkChunkTiles];
    const int m = blockIdx.y;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t c0 = (static_cast<int64_t>(blockIdx.x) * (kBlock / 64) + wave) * kScanChunksPerWave;
    if (c0 >= n_chunks) return;  // whole waves: no barrier below spans waves
    uint32_t *sel = sel_all[wave];
    const TopkRow r = rows[m];
    uint32_t cnt[kScanChunksPerWave];
    uint2 run[kScanChunksPerWave];
#pragma unroll
    for (int q = 0; q < kScanChunksPerWave; ++q) {
        const int64_t c = c0 + q;
        const int64_t t = c * kTopkChunkTiles + lane;
        cnt[q] = (c < n_chunks && t < n_tiles) ? tile_cnt[static_cast<int64_t>(m) * n_tiles + t] : 0u;
        run[q] = c < n_chunks ? runs[static_cast<int64_t>(m) * n_chunks + c] : make_uint2(0u, 0u);
    }
    const uint32_t *krow = ckey + static_cast<int64_t>(m) * cap;
    const uint32_t *irow = cidx + static_cast<int64_t>(m) * cap;
#pragma unroll
    for (int q = 0; q < kScanChunksPerWave; ++q) {
        const int64_t c = c0 + q;
        if (c >= n_chunks) break;  // uniform
        const int64_t t = c * kTopkChunkTiles + lane;
        uint32_t n_here = cnt[q];
        if (!r.fallback) {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            sel[lane] = 0u;
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            const int64_t first_tile = c * kTopkChunkTiles;
            // up to 8 of the lane's candidates loaded at once (a run holds at
            // most 1024)
            constexpr int kRunU = 8;
            for (uint32_t j0 = lane; j0 < run[q].y; j0 += 64 * kRunU) {
                uint2 cd[kRunU];
#pragma unroll
                for (int u = 0; u < kRunU; ++u) {
                    const uint32_t j = j0 + 64 * u;
                    const int64_t pos = static_cast<int64_t>(run[q].x) + j;
                    cd[u] = (j < run[q].y && pos < cap) ? make_uint2(krow[pos], irow[pos]) : make_uint2(0u, 0xFFFFFFFFu);
                }
#pragma unroll
                for (int u = 0; u < kRunU; ++u) {
                    if (j0 + 64 * u >= run[q].y) continue;
                    if (cd[u].x > r.T || (cd[u].x == r.T && cd[u].y <= r.I)) {
                        const int64_t lt = static_cast<int64_t>(cd[u].y / kTopkTile) - first_tile;
                        if (lt >= 0 && lt < kTopkChunkTiles) atomicAdd(&sel[lt], 1u);
                    }
                }
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            n_here += sel[lane];
        }
        const uint32_t incl = wave_incl_scan(n_here);
        if (t < n_tiles) tile_off[static_cast<int64_t>(m) * n_tiles + t] = static_cast<uint16_t>(incl - n_here);
        if (lane == 63) chunk_sum[static_cast<int64_t>(m) * n_chunks + c] = incl;
    }
}

// 8. Exclusive scan of the chunk totals of each row (one workgroup per row).
__global__ __launch_bounds__(1024) void k_topk_chunk_scan(TopkRow *__restrict__ rows,
                                                          const uint32_t *__restrict__ chunk_sum,
                                                          uint32_t *__restrict__ chunk_off, int64_t n_chunks) {
    __shared__ uint32_t wsum[16];
    const int m = blockIdx.x;
    const uint32_t *src = chunk_sum + static_cast<int64_t>(m) * n_chunks;
    uint32_t *dst = chunk_off + static_cast<int64_t>(m) * n_chunks;
    uint32_t carry = 0;
    for (int64_t c0 = 0; c0 < n_chunks; c0 += 1024) {
        const int64_t c = c0 + threadIdx.x;
        const uint32_t v = c < n_chunks ? src[c] : 0u;
        uint32_t total;
        const uint32_t ex = block_exclusive_scan(v, wsum, total);
        if (c < n_chunks) dst[c] = carry + ex;
        carry += total;
        __syncthreads();  // wsum is reused by the next round's scan
    }
    if (threadIdx.x == 0) rows[m].total = carry;
}

// Server side: scatter the messages to the dense p-hat (unpack); indices at
// or beyond d (only a malformed message has them) are skipped.
__global__ __launch_bounds__(kBlock) void k_topk_scatter(const float *__restrict__ val, const uint32_t *__restrict__ idx,
                                                         int64_t k, int64_t d, float *__restrict__ out, int64_t ld) {
    const int m = blockIdx.y;
    for (int64_t j = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x; j < k;
         j += static_cast<int64_t>(gridDim.x) * kBlock) {
        const uint32_t i = idx[static_cast<int64_t>(m) * k + j];
        if (i < d) out[static_cast<int64_t>(m) * ld + i] = val[static_cast<int64_t>(m) * k + j];
    }
}

// Server average of the M top-k messages by column tiles: the average of
// the decoded messages, summed in ascending worker order in binary32.  Each
// worker's list is sorted by index, so its entries in tile T are one run
// [start(T, m), start(T + 1, m)).  Each thread of a workgroup owns kAggCols
// columns of the tile (4 consecutive in each half) and carries their sums in
// registers across the groups of 64 workers.  A group takes one of two
// routes:
//  - sparse (at most kAggStage entries): every run is staged in LDS and each
//    staged entry sets its worker's bit in its column's 64-bit mask; a scan
//    of the columns' entry counts places each entry at its column's first
//    position plus the number of lower workers in the mask; each thread then
//    adds its columns' entries in that order;
//  - dense: rounds of kAggDenseRows workers.  A round's runs are read in
//    aligned 16-byte chunks and scattered to one LDS row per worker (a
//    column without an entry holds +0); each thread adds its columns of the
//    rows in worker order, then clears them.  A round's first chunks are
//    loaded two rounds ahead, into one of two sets of registers.
// The sums start from -0: fl(-0 + x) = x for every x, so starting there
// gives the definition's sum, which starts from worker 0's term.  In round
// to nearest a partial sum is -0 exactly while every term so far is -0, and
// adding +0 changes a partial sum only when it is -0 (to +0).  So the +0
// terms of workers without an entry can be added at any point of the chain:
// the dense route adds them in place (cleared row entries), the sparse
// route adds one +0 for a column that a worker of the group did not send.
// Indices outside the tile, and runs longer than the tile (only a malformed
// message has them), are skipped and cut to the tile's width.
constexpr int kAggTile = 2048;      // columns per tile
constexpr int kAggHalf = kAggTile / 2;
constexpr int kAggStage = 1536;     // entries of a group staged on the sparse route
constexpr int kAggGroup = 64;       // workers per group: the bits of a column mask
constexpr int kAggCols = kAggTile / kBlock;  // columns per thread
constexpr int kAggDenseRows = 4;    // workers per round on the dense route
constexpr int kAggSparseU = 2;      // 16-byte chunks per thread and load on the sparse route
constexpr int kAggDenseU = 1;       // ... and on the dense route, which keeps two such loads in flight
constexpr int kAggStrip = 4;        // tiles per workgroup (see agg_tile_of)
static_assert(kAggCols == 8 && kAggHalf == 4 * kBlock, "each thread's columns are one float4 per half");

// column i (0..7) of thread t: 4t + i in the first half, 1024 + 4t + i - 4 in the second
__device__ __forceinline__ int agg_col(int t, int i) { return (i < 4 ? 0 : kAggHalf - 4) + 4 * t + i; }

// start(T, m) = the first entry j of worker m with idx[j] >= T * kAggTile,
// for T = 0 .. n_t (k for the tiles past the last entry), stored [T][M] so
// that a tile's M starts are contiguous.  Entry j starts the tiles
// (tile(j - 1), tile(j)] (tile(-1) = -1; entry k stands for the end, in
// tile n_t).  The lists are read in aligned 16-byte chunks of the flat
// [M][k] array: a wave takes kStartsLoads * 64 consecutive chunks of a row
// in coalesced rounds (round u: chunk u * 64 + lane), all loaded before the
// first is examined; a chunk's entries outside the row are not the row's.
// A round whose last entry lies in the tile of the entry before the round
// starts nothing (sorted lists) and is passed over.  Otherwise each lane
// writes the starts of its own entries (an entry after a run of empty tiles
// starts all of them), except a lane with more than kStartsLongRun to write,
// whose starts the whole wave writes.
constexpr int kStartsLoads = 4;
constexpr int kStartsLongRun = 8;  // more starts than this per lane and round: written by the wave

__device__ __forceinline__ uint32_t u4_at(const uint4 &v, int i) {
    return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

__global__ __launch_bounds__(kBlock) void k_topk_agg_starts(const uint32_t *__restrict__ idx, int64_t k, int32_t M,
                                                            int32_t n_t, uint32_t *__restrict__ start) {
    // Workgroup b takes segment b / M of a row.  The M workgroups of a
    // segment are consecutive, and with M a multiple of 8 the XCD of b
    // (b % 8) takes M / 8 consecutive rows: a tile's M starts are written
    // close in time, each contiguous eighth of them from one L2, which merges
    // the 4-byte stores before they reach HBM.
    const uint32_t b = blockIdx.x, um = static_cast<uint32_t>(M);
    const uint32_t useg = b / um;
    const int seg = static_cast<int>(useg), t = static_cast<int>(b - useg * um);
    const int m = M % 8 == 0 ? (t % 8) * (M / 8) + t / 8 : t;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t row0 = static_cast<int64_t>(m) * k;  // flat index of the row's first entry
    const int64_t c_first = row0 >> 2;
    const int64_t c_last = (row0 + k - 1) >> 2;               // the last chunk holding an entry of the row
    const int64_t n_ch = ((row0 + k) >> 2) - c_first + 1;     // ... and the chunk of the end (entry k)
    const int64_t cw = (static_cast<int64_t>(seg) * (kBlock / 64) + wave) * (64 * kStartsLoads);
    if (cw >= n_ch) return;
    const uint4 *chunks = reinterpret_cast<const uint4 *>(idx);
    uint4 v[kStartsLoads];
#pragma unroll
    for (int u = 0; u < kStartsLoads; ++u) {
        const int64_t c = c_first + cw + 64 * u + lane;
        v[u] = chunks[c < c_last ? c : c_last];
    }
    // the tile of an entry: -1 before the row, n_t for the end and past it
    auto tile_of = [&](int64_t j, uint32_t x) -> int {
        return j < 0 ? -1 : j < k ? min(static_cast<int>(x / kAggTile), n_t) : n_t;
    };
    const int64_t j_wave = 4 * (c_first + cw) - row0;  // the wave's first entry (row-relative)
    int t_before = j_wave - 1 >= 0 ? tile_of(j_wave - 1, idx[row0 + j_wave - 1]) : -1;
    // every entry the wave loaded lies in the row (all waves but the first
    // and last of a row): the tile is the index's alone
    const bool inside = j_wave >= 0 && j_wave + 4 * 64 * kStartsLoads <= k;
#pragma unroll
    for (int u = 0; u < kStartsLoads; ++u) {
        const int64_t j0 = j_wave + 4 * (64 * u + lane);  // row-relative index of the chunk's entry 0
        int t[4];
        if (inside) {
#pragma unroll
            for (int i = 0; i < 4; ++i) t[i] = min(static_cast<int>(u4_at(v[u], i) / kAggTile), n_t);
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) t[i] = tile_of(j0 + i, u4_at(v[u], i));
        }
        const int t_round_last = __builtin_amdgcn_readlane(t[3], 63);
        if (t_round_last == t_before) continue;  // no entry of the round starts a tile
        // the tile of the previous lane's last entry (DPP shift right by one
        // lane across the wave; lane 0 keeps t_before, the tile of the entry
        // before the round)
        int n[4];
        int tp = __builtin_amdgcn_update_dpp(t_before, t[3], 0x138, 0xF, 0xF, false);
        int n_lane = 0;  // the tiles this lane's four entries start
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            n[i] = t[i] > tp ? t[i] - tp : 0;
            n_lane += n[i];
            tp = t[i] > tp ? t[i] : tp;
        }
        t_before = t_round_last;
        // Each lane writes the starts of its own entries, entry j0 + i those of
        // tiles t[i] - n[i] + 1 .. t[i], except a lane that starts a long run
        // of empty tiles: the wave writes that lane's starts together, 64 at a
        // time, one such lane after the other.
        const uint64_t lng = __ballot(n_lane > kStartsLongRun);
        if (n_lane <= kStartsLongRun) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                for (int q = 0; q < n[i]; ++q)
                    start[static_cast<int64_t>(t[i] - q) * M + m] = static_cast<uint32_t>(j0 + i);
        }
        for (uint64_t rest = lng; rest != 0; rest &= rest - 1) {
            const int L = __builtin_ctzll(rest);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int nl = __builtin_amdgcn_readlane(n[i], L);
                const int tl = __builtin_amdgcn_readlane(t[i], L);
                const uint32_t jl = static_cast<uint32_t>(j_wave + 4 * (64 * u + L) + i);
                for (int q = lane; q < nl; q += 64) start[static_cast<int64_t>(tl - q) * M + m] = jl;
            }
        }
    }
}

// A barrier that orders LDS only: outstanding global loads stay in flight.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

union AggLds {
    struct {
        unsigned long long mask[kAggTile];  // bit w: worker g0 + w has an entry in the column
        uint16_t col_base[kAggTile];        // first position of the column's entries in `placed`
        uint16_t st_col[kAggStage];         // staged entries: column (0xFFFF: outside the tile),
        uint8_t st_w[kAggStage];            //   worker within the group,
        float st_val[kAggStage];            //   value
        float placed[kAggStage];            // the values in (column, worker) order
    } s;
    float rows[kAggDenseRows][kAggTile];    // dense route: one row per worker of a round
};

// A group's runs as both routes read them: worker w's run starts at
// entry G0 = (g0 + w) * k + start of the flat [M][k] lists; its chunks are
// the 16-byte words c0 .. c0 + nc - 1 with c0 = G0 / 4, and the run's first
// entry is entry lo = G0 % 4 of chunk c0.  ch_off is the exclusive prefix of
// the chunk counts over the group.
struct AggRuns {
    uint32_t woff[kAggGroup + 1];  // exclusive prefix of the run lengths
    unsigned long long ch_c0[kAggGroup];
    uint32_t ch_off[kAggGroup + 1];
    uint32_t ch_lo[kAggGroup];
};

// Chunks of one load of the dense route: chunk q0 + tid + kBlock * u of the
// round's workers w0 .. w1 - 1 (their chunks ch_off[w0] .. ch_off[w1]),
// with a 4-bit mask of the entries that belong to the run and the row.
struct DenseChunks {
    uint4 idx[kAggDenseU];
    f32x4 val[kAggDenseU];
    uint32_t tag[kAggDenseU];  // bits 0..3: entries of the run; bits 4..: row of the round
};

__device__ __forceinline__ void agg_dense_load(DenseChunks &L, const float *__restrict__ val,
                                               const uint32_t *__restrict__ idx, const AggRuns &R, int w0, int w1,
                                               uint32_t q0) {
    const uint32_t a = R.ch_off[w0], e = R.ch_off[w1];
    uint32_t o[kAggDenseRows];  // o[j]: the first chunk of row j (rows past w1 start at the end)
#pragma unroll
    for (int j = 1; j < kAggDenseRows; ++j) o[j] = R.ch_off[w0 + j < w1 ? w0 + j : w1];
#pragma unroll
    for (int u = 0; u < kAggDenseU; ++u) {
        const uint32_t Q0 = a + q0 + threadIdx.x + kBlock * u;
        const bool live = Q0 < e;
        const uint32_t Q = live ? Q0 : a;  // past the end: the round's first chunk, masked out
        int r = 0;
#pragma unroll
        for (int j = 1; j < kAggDenseRows; ++j) r += Q >= o[j];
        const int w = w0 + r;
        const uint32_t ql = Q - R.ch_off[w];
        const unsigned long long c = R.ch_c0[w] + ql;
        L.idx[u] = reinterpret_cast<const uint4 *>(idx)[c];
        L.val[u] = reinterpret_cast<const f32x4 *>(val)[c];
        const int rel = static_cast<int>(4 * ql) - static_cast<int>(R.ch_lo[w]);
        const int n = static_cast<int>(R.woff[w + 1] - R.woff[w]);
        uint32_t m4 = 0u;
#pragma unroll
        for (int i = 0; i < 4; ++i) m4 |= (live && rel + i >= 0 && rel + i < n) ? (1u << i) : 0u;
        L.tag[u] = m4 | (static_cast<uint32_t>(r) << 4);
    }
}

__device__ __forceinline__ void agg_dense_scatter(const DenseChunks &L, AggLds &S, uint32_t base_lo, bool addressable) {
#pragma unroll
    for (int u = 0; u < kAggDenseU; ++u) {
        float *row = S.rows[L.tag[u] >> 4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t c = (i == 0 ? L.idx[u].x : i == 1 ? L.idx[u].y : i == 2 ? L.idx[u].z : L.idx[u].w) - base_lo;
            if (((L.tag[u] >> i) & 1u) && addressable && c < static_cast<uint32_t>(kAggTile)) row[c] = elem(L.val[u], i);
        }
    }
}

// Chunks of one load of the sparse route: chunk q0 + tid + kBlock * u of
// the whole group (chunks 0 .. ch_off[gn]), with the stage position of the
// chunk's entry 0 and a 4-bit mask of the entries that belong to the run.
struct SparseChunks {
    uint4 idx[kAggSparseU];
    f32x4 val[kAggSparseU];
    int pos[kAggSparseU];       // stage position of entry 0 (entries 1..3 follow)
    uint32_t tag[kAggSparseU];  // bits 0..3: entries of the run; bits 4..: worker in the group
};

__device__ __forceinline__ void agg_sparse_load(SparseChunks &L, const float *__restrict__ val,
                                                const uint32_t *__restrict__ idx, const AggRuns &R, int gn,
                                                uint32_t q0) {
    const uint32_t e = R.ch_off[gn];
#pragma unroll
    for (int u = 0; u < kAggSparseU; ++u) {
        const uint32_t Q0 = q0 + threadIdx.x + kBlock * u;
        const bool live = Q0 < e;
        const uint32_t Q = live ? Q0 : 0u;  // past the end: the group's first chunk, masked out
        int lo = 0, hi = gn - 1;            // the last worker whose first chunk is <= Q
        while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if (R.ch_off[mid] <= Q) lo = mid;
            else hi = mid - 1;
        }
        const uint32_t ql = Q - R.ch_off[lo];
        const unsigned long long c = R.ch_c0[lo] + ql;
        L.idx[u] = reinterpret_cast<const uint4 *>(idx)[c];
        L.val[u] = reinterpret_cast<const f32x4 *>(val)[c];
        const int rel = static_cast<int>(4 * ql) - static_cast<int>(R.ch_lo[lo]);
        const int n = static_cast<int>(R.woff[lo + 1] - R.woff[lo]);
        uint32_t m4 = 0u;
#pragma unroll
        for (int i = 0; i < 4; ++i) m4 |= (live && rel + i >= 0 && rel + i < n) ? (1u << i) : 0u;
        L.pos[u] = static_cast<int>(R.woff[lo]) + rel;
        L.tag[u] = m4 | (static_cast<uint32_t>(lo) << 4);
    }
}

// Tile s of workgroup b's strip.  Workgroups go to the 8 XCDs in turn
// (b % 8) and tiles go to them in blocks of 8 consecutive tiles (block j on
// XCD j % 8), so that neighbouring tiles, which share the cache lines at
// their runs' ends and a row of the start table, meet in one L2.  Within
// an XCD, its i-th workgroup takes the XCD's tiles i, i + per, i + 2 per ...
// (per = grid / 8), which spreads the dense bands over the workgroups.
__device__ __forceinline__ int64_t agg_tile_of(int64_t b, int s, int64_t grid) {
    const int64_t x = b % 8, i = b / 8, per = grid / 8;
    const int64_t z = i + static_cast<int64_t>(s) * per;
    return 64 * (z / 8) + 8 * x + (z % 8);
}

// four workgroups per CU: at most 128 VGPRs and 40 KB of LDS each
__global__ __launch_bounds__(kBlock, 4) void k_topk_agg_tiles(const float *__restrict__ val,
                                                           const uint32_t *__restrict__ idx, int64_t k, int32_t M,
                                                           const uint32_t *__restrict__ start, int64_t n_t,
                                                           int64_t d, int64_t ld, float *__restrict__ Qhat,
                                                           float invM) {
    __shared__ AggLds S;
    __shared__ AggRuns R;
    __shared__ uint32_t wsum[kBlock / 64];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int n_groups = (M + kAggGroup - 1) / kAggGroup;
    const int n_it = kAggStrip * n_groups;  // (tile, group) pairs of this workgroup
    // Every wave reads the starts itself, so that each knows a tile's entry
    // count without LDS; with one group they are read for the whole strip
    // up front.
    uint32_t ss[kAggStrip], ee[kAggStrip];
    if (n_groups == 1) {
#pragma unroll
        for (int q = 0; q < kAggStrip; ++q) {
            const int64_t T = agg_tile_of(blockIdx.x, q, gridDim.x);
            ss[q] = ee[q] = 0u;
            if (T < n_t && lane < M) {
                ss[q] = start[T * M + lane];
                ee[q] = start[(T + 1) * M + lane];
            }
        }
    }
    float acc[kAggCols];
    for (int it = 0; it < n_it; ++it) {
        const int sq = it / n_groups;
        const int64_t T = agg_tile_of(blockIdx.x, sq, gridDim.x);
        if (T >= n_t) break;  // uniform: the strip's later tiles are past the end too
        const int g0 = (it % n_groups) * kAggGroup;
        const int gn = M - g0 < kAggGroup ? M - g0 : kAggGroup;
        const int64_t base = T * kAggTile;
        if (g0 == 0) {
#pragma unroll
            for (int i = 0; i < kAggCols; ++i) acc[i] = -0.0f;
        }
        uint32_t s_raw = 0u, e_raw = 0u;
        if (n_groups == 1) {
#pragma unroll
            for (int q = 0; q < kAggStrip; ++q)
                if (q == sq) {
                    s_raw = ss[q];
                    e_raw = ee[q];
                }
        } else if (lane < gn) {
            s_raw = start[T * M + g0 + lane];
            e_raw = start[(T + 1) * M + g0 + lane];
        }
        const int64_t s0 = min(static_cast<int64_t>(s_raw), k);
        const int64_t e0 = min(static_cast<int64_t>(e_raw), k);
        const uint32_t rn = e0 > s0 ? static_cast<uint32_t>(min(e0 - s0, static_cast<int64_t>(kAggTile))) : 0u;
        const uint32_t incl = wave_incl_scan(rn);
        const uint32_t total = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(incl), 63));
        if (total == 0u) {
#pragma unroll
            for (int i = 0; i < kAggCols; ++i) acc[i] = add_rn(acc[i], 0.0f);  // the group's terms are +0
        } else {
            // the group's runs, their offsets and chunks, for every wave (wave 0 writes them)
            if (wave == 0) {
                const unsigned long long G0 = static_cast<unsigned long long>(g0 + lane) * static_cast<unsigned long long>(k) +
                                              static_cast<unsigned long long>(s0);
                const unsigned long long c0 = G0 >> 2;
                const uint32_t nc = rn ? static_cast<uint32_t>(((G0 + rn + 3) >> 2) - c0) : 0u;
                const uint32_t cincl = wave_incl_scan(nc);
                R.woff[lane] = incl - rn;
                R.ch_c0[lane] = c0;
                R.ch_off[lane] = cincl - nc;
                R.ch_lo[lane] = static_cast<uint32_t>(G0 & 3u);
                if (lane == 63) {
                    R.woff[kAggGroup] = incl;
                    R.ch_off[kAggGroup] = cincl;
                }
            }
            lds_barrier();
            const uint32_t base_lo = static_cast<uint32_t>(base);
            const bool addressable = (static_cast<unsigned long long>(base) >> 32) == 0;  // idx is 32-bit
            if (total <= kAggStage) {
                for (int c = tid; c < kAggTile; c += kBlock) S.s.mask[c] = 0ull;
                lds_barrier();
                // stage every run and mark each entry's worker in its column
                for (uint32_t q0 = 0; q0 < R.ch_off[gn]; q0 += kBlock * kAggSparseU) {
                    SparseChunks L;
                    agg_sparse_load(L, val, idx, R, gn, q0);
#pragma unroll
                    for (int u = 0; u < kAggSparseU; ++u) {
                        const uint32_t w = L.tag[u] >> 4;
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            if (!((L.tag[u] >> i) & 1u)) continue;
                            const uint32_t c = u4_at(L.idx[u], i) - base_lo;
                            const bool in = addressable && c < static_cast<uint32_t>(kAggTile);
                            const int g = L.pos[u] + i;
                            S.s.st_col[g] = in ? static_cast<uint16_t>(c) : static_cast<uint16_t>(0xFFFFu);
                            S.s.st_val[g] = elem(L.val[u], i);
                            S.s.st_w[g] = static_cast<uint8_t>(w);
                            if (in) atomicOr(&S.s.mask[c], 1ull << w);
                        }
                    }
                }
                lds_barrier();
                // each column's first position: exclusive scan of the entry counts
                uint32_t cnt[kAggCols], mine = 0u;
#pragma unroll
                for (int i = 0; i < kAggCols; ++i) {
                    cnt[i] = static_cast<uint32_t>(__popcll(S.s.mask[agg_col(tid, i)]));
                    mine += cnt[i];
                }
                const uint32_t incl = wave_incl_scan(mine);
                if (lane == 63) wsum[wave] = incl;
                lds_barrier();
                uint32_t pos = incl - mine;
                for (int w = 0; w < wave; ++w) pos += wsum[w];
#pragma unroll
                for (int i = 0; i < kAggCols; ++i) {
                    S.s.col_base[agg_col(tid, i)] = static_cast<uint16_t>(pos);
                    pos += cnt[i];
                }
                lds_barrier();
                // each entry to its place: the column's first position plus the
                // number of lower workers with an entry in the column
                for (uint32_t g = tid; g < total; g += kBlock) {
                    const uint32_t c = S.s.st_col[g];
                    if (c == 0xFFFFu) continue;
                    const unsigned long long below = (1ull << S.s.st_w[g]) - 1ull;
                    S.s.placed[S.s.col_base[c] + __popcll(S.s.mask[c] & below)] = S.s.st_val[g];
                }
                lds_barrier();
                // the columns' sums in ascending worker order
#pragma unroll
                for (int i = 0; i < kAggCols; ++i) {
                    const uint32_t b = S.s.col_base[agg_col(tid, i)];
                    for (uint32_t q = 0; q < cnt[i]; ++q) acc[i] = add_rn(acc[i], S.s.placed[b + q]);
                    if (cnt[i] != static_cast<uint32_t>(gn)) acc[i] = add_rn(acc[i], 0.0f);  // an absent worker's +0
                }
            } else {
                // the rows start cleared; each thread clears its own columns
                const f32x4 zero = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
                for (int r = 0; r < kAggDenseRows; ++r) {
                    st4(&S.rows[r][4 * tid], zero);
                    st4(&S.rows[r][kAggHalf + 4 * tid], zero);
                }
                const int n_rounds = (gn + kAggDenseRows - 1) / kAggDenseRows;
                // two sets of chunk registers: round r's first chunks are
                // loaded during round r - 2
                DenseChunks La, Lb;
                auto load = [&](DenseChunks &L, int w0, uint32_t q0) {
                    const int w1 = w0 + kAggDenseRows < gn ? w0 + kAggDenseRows : gn;
                    if (w0 < gn && R.ch_off[w1] - R.ch_off[w0] > q0) {
                        agg_dense_load(L, val, idx, R, w0, w1, q0);
                    } else {
#pragma unroll
                        for (int u = 0; u < kAggDenseU; ++u) L.tag[u] = 0u;
                    }
                };
                auto round = [&](DenseChunks &L, int r) {
                    const int w0 = r * kAggDenseRows;
                    const int w1 = w0 + kAggDenseRows < gn ? w0 + kAggDenseRows : gn;
                    const uint32_t nch = R.ch_off[w1] - R.ch_off[w0];
                    agg_dense_scatter(L, S, base_lo, addressable);
                    for (uint32_t q0 = kBlock * kAggDenseU; q0 < nch; q0 += kBlock * kAggDenseU) {
                        load(L, w0, q0);
                        agg_dense_scatter(L, S, base_lo, addressable);
                    }
                    if (r + 2 < n_rounds) load(L, w0 + 2 * kAggDenseRows, 0u);
                    lds_barrier();
                    for (int rr = 0; rr < w1 - w0; ++rr) {
                        const f32x4 x0 = ld4(&S.rows[rr][4 * tid]), x1 = ld4(&S.rows[rr][kAggHalf + 4 * tid]);
#pragma unroll
                        for (int c = 0; c < 4; ++c) {
                            acc[c] = add_rn(acc[c], elem(x0, c));
                            acc[c + 4] = add_rn(acc[c + 4], elem(x1, c));
                        }
                        st4(&S.rows[rr][4 * tid], zero);
                        st4(&S.rows[rr][kAggHalf + 4 * tid], zero);
                    }
                    lds_barrier();
                };
                load(La, 0, 0u);
                load(Lb, kAggDenseRows, 0u);
                lds_barrier();  // the rows are cleared before the first scatter
                for (int r = 0; r < n_rounds; r += 2) {
                    round(La, r);
                    if (r + 1 < n_rounds) round(Lb, r + 1);
                }
            }
            lds_barrier();  // the next pair rewrites the group's tables and the LDS buffers
        }
        if (g0 + gn == M) {
            // ld is a multiple of 1024: a half's four columns are all inside or all outside
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int64_t col = base + h * kAggHalf + 4 * tid;
                if (col < ld) {
                    f32x4 q;
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        const float sacc = acc[4 * h + c];
                        set_elem(q, c, col + c >= d ? 0.0f
                                       : invM > 0.0f ? mul_rn(sacc, invM)
                                                     : static_cast<float>(static_cast<double>(sacc) /
                                                                          static_cast<double>(M)));
                    }
                    st4(Qhat + col, q);
                }
            }
        }
    }
}

unsigned grid_for(int64_t n, int64_t cap_blocks = 65536) {
    int64_t b = (n + kBlock - 1) / kBlock;
    if (b < 1) b = 1;
    return static_cast<unsigned>(b < cap_blocks ? b : cap_blocks);
}

}  // namespace

hipError_t topk_alloc(dqgan_plan_s &P) {
    TopkScratch &S = P.topk;
    const dqgan_desc &D = P.desc;
    S.n_tiles = D.ld / kTopkTile;
    S.n_chunks = (S.n_tiles + kTopkChunkTiles - 1) / kTopkChunkTiles;
    S.n_sample_chunks = (D.d + kSampleStride - 1) / kSampleStride;
    int64_t ns = 0;
    for (int64_t c = 0; c < S.n_sample_chunks; ++c) {
        const int64_t a = c * kSampleStride;
        ns += (D.d - a < kTopkTile) ? D.d - a : kTopkTile;
    }
    S.n_samples = static_cast<uint32_t>(ns);
    int64_t cap = D.k > 65536 ? D.k : 65536;
    S.cap = cap < D.d ? cap : D.d;
    const size_t M = static_cast<size_t>(D.M);
    const size_t digit_words = M * kSelectPasses * kDigitBins;
    hipError_t e = hipMalloc(reinterpret_cast<void **>(&S.rows), M * sizeof(TopkRow));
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&S.ctr), M * kRowCtrWords * sizeof(uint32_t));
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&S.hist), M * kSampleBins * sizeof(uint32_t));
    // the sample histogram starts at zero; every iteration zeroes it again once read
    if (e == hipSuccess) e = hipMemset(S.hist, 0, M * kSampleBins * sizeof(uint32_t));
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&S.sel_hist), M * kDigitBins * sizeof(uint32_t));
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&S.fb_hist), digit_words * sizeof(uint32_t));
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&S.cand), M * static_cast<size_t>(S.cap) * sizeof(uint2));
    if (e == hipSuccess)
        e = hipMalloc(reinterpret_cast<void **>(&S.play), M * static_cast<size_t>(S.cap) * sizeof(uint2));
    if (e == hipSuccess)
        e = hipMalloc(reinterpret_cast<void **>(&S.runs), M * static_cast<size_t>(S.n_chunks) * sizeof(uint2));
    if (e == hipSuccess)
        e = hipMalloc(reinterpret_cast<void **>(&S.tile_cnt), M * static_cast<size_t>(S.n_tiles) * sizeof(uint16_t));
    if (e == hipSuccess)
        e = hipMalloc(reinterpret_cast<void **>(&S.tile_off), M * static_cast<size_t>(S.n_tiles) * sizeof(uint16_t));
    if (e == hipSuccess)
        e = hipMalloc(reinterpret_cast<void **>(&S.chunk_sum), M * static_cast<size_t>(S.n_chunks) * sizeof(uint32_t));
    if (e == hipSuccess)
        e = hipMalloc(reinterpret_cast<void **>(&S.chunk_off), M * static_cast<size_t>(S.n_chunks) * sizeof(uint32_t));
    S.n_agg_tiles = (D.ld + kAggTile - 1) / kAggTile;
    if (e == hipSuccess)
        e = hipMalloc(reinterpret_cast<void **>(&S.agg_start),
                      M * static_cast<size_t>(S.n_agg_tiles + 1) * sizeof(uint32_t));
    if (e == hipSuccess) e = hipDeviceSynchronize();  // the memset is done before the plan is used
    return e;
}

void topk_free(dqgan_plan_s &P) {
    TopkScratch &S = P.topk;
    (void)hipFree(S.rows);
    (void)hipFree(S.ctr);
    (void)hipFree(S.hist);
    (void)hipFree(S.sel_hist);
    (void)hipFree(S.fb_hist);
    (void)hipFree(S.cand);
    (void)hipFree(S.play);
    (void)hipFree(S.runs);
    (void)hipFree(S.tile_cnt);
    (void)hipFree(S.tile_off);
    (void)hipFree(S.chunk_sum);
    (void)hipFree(S.chunk_off);
    (void)hipFree(S.agg_start);
    S = TopkScratch{};
}

hipError_t launch_topk_select(const dqgan_plan_s &P, float eta, const float *G, const float *E, hipStream_t st) {
    const TopkScratch &S = P.topk;
    const dqgan_desc &D = P.desc;
    const unsigned M = static_cast<unsigned>(D.M);
    // the candidate lists: a key plane [M][cap], then an index plane [M][cap]
    uint32_t *ckey = reinterpret_cast<uint32_t *>(S.cand);
    uint32_t *cidx = ckey + static_cast<int64_t>(D.M) * S.cap;
    const int64_t sb = (S.n_sample_chunks + kSampleThreads / 64 - 1) / (kSampleThreads / 64);
    hipLaunchKernelGGL(k_topk_sample, dim3(static_cast<unsigned>(sb < kSampleBlocks ? sb : kSampleBlocks), M),
                       dim3(kSampleThreads), 0, st,
                       G, E, eta, D.d, D.ld, S.n_sample_chunks, S.hist);
    hipLaunchKernelGGL(k_topk_band, dim3(M), dim3(1024), 0, st, S.hist, S.sel_hist, S.rows, S.ctr, S.n_samples, D.d,
                       D.k);
    hipLaunchKernelGGL(k_topk_pass, dim3(static_cast<unsigned>(S.n_chunks), M), dim3(kBlock), 0, st, G, E, eta, D.d,
                       D.ld, S.n_tiles, S.rows, S.ctr, S.tile_cnt, ckey, cidx, S.cap, S.runs, S.n_chunks);
    hipLaunchKernelGGL(k_topk_sel_top, dim3(kSelBlocks, M), dim3(kBlock), 0, st, S.rows, S.ctr, ckey, S.cap, D.k,
                       S.sel_hist);
    hipLaunchKernelGGL(k_topk_sel_collect, dim3(kSelBlocks, M), dim3(kBlock), 0, st, S.rows, S.ctr, ckey, cidx,
                       S.cap, D.k, S.sel_hist, S.play);
    hipLaunchKernelGGL(k_topk_sel_finish, dim3(M), dim3(1024), 0, st, S.rows, S.ctr, S.cap, D.k, S.sel_hist, S.play,
                       S.fb_hist);
    for (int pass = 0; pass < kSelectPasses; ++pass)
        hipLaunchKernelGGL(k_topk_fb_hist, dim3(kFbBlocks), dim3(kBlock), 0, st, pass, G, E, eta, D.d, D.ld, D.M, D.k,
                           S.rows, S.fb_hist);
    hipLaunchKernelGGL(k_topk_fb_recount, dim3(256), dim3(kBlock), 0, st, G, E, eta, D.d, D.ld, S.n_tiles, D.M, D.k,
                       S.rows, S.fb_hist, S.tile_cnt);
    hipLaunchKernelGGL(k_topk_spill_count, dim3(kSpillBlocks, M), dim3(kBlock), 0, st, S.rows, ckey, cidx, S.cap,
                       S.tile_cnt, S.n_tiles);
    const int64_t scan_per_block = (kBlock / 64) * kScanChunksPerWave;
    hipLaunchKernelGGL(k_topk_count_scan, dim3(static_cast<unsigned>((S.n_chunks + scan_per_block - 1) / scan_per_block), M),
                       dim3(kBlock), 0, st,
                       S.rows, ckey, cidx,
                       S.cap, S.runs, S.tile_cnt, S.tile_off, S.chunk_sum, S.n_tiles, S.n_chunks);
    hipLaunchKernelGGL(k_topk_chunk_scan, dim3(M), dim3(1024), 0, st, S.rows, S.chunk_sum, S.chunk_off, S.n_chunks);
    return hipGetLastError();
}

hipError_t launch_topk_compress(const dqgan_plan_s &P, float eta, const float *G, float *E, const dqgan_wire &w,
                                hipStream_t st) {
    hipError_t e = launch_topk_select(P, eta, G, E, st);
    if (e != hipSuccess) return e;
    return launch_topk_encode_rows(P, eta, G, E, w, st);
}

hipError_t launch_topk_unpack(const dqgan_plan_s &P, const dqgan_wire &w, float *Phat, hipStream_t st) {
    const dqgan_desc &D = P.desc;
    const int64_t n = static_cast<int64_t>(D.M) * D.ld;
    hipLaunchKernelGGL(k_fill_f32, dim3(grid_for(n)), dim3(kBlock), 0, st, Phat, n);
    hipLaunchKernelGGL(k_topk_scatter, dim3(grid_for(D.k, 4096), static_cast<unsigned>(D.M)), dim3(kBlock), 0, st,
                       w.val, w.idx, D.k, D.d, Phat, D.ld);
    return hipGetLastError();
}

hipError_t launch_topk_aggregate(const dqgan_plan_s &P, const dqgan_wire &w, float *Qhat, hipStream_t st) {
    const dqgan_desc &D = P.desc;
    const TopkScratch &S = P.topk;
    // a row spans at most k / 4 + 2 chunks, its end included
    const int64_t per_block = static_cast<int64_t>(kBlock) * kStartsLoads;
    const int64_t sb = (D.k / 4 + 2 + per_block - 1) / per_block;
    hipLaunchKernelGGL(k_topk_agg_starts, dim3(static_cast<unsigned>(sb * D.M)), dim3(kBlock), 0,
                       st, w.idx, D.k, D.M, static_cast<int32_t>(S.n_agg_tiles), S.agg_start);
    const float im = (D.M & (D.M - 1)) == 0 ? 1.0f / static_cast<float>(D.M) : 0.0f;
    // 8 x per workgroups, per large enough that every tile's place in its
    // XCD's list (at most n_t / 8 + 7) is inside a strip
    const int64_t per = (S.n_agg_tiles / 8 + 8 + kAggStrip - 1) / kAggStrip;
    const int64_t nb = 8 * per;
    hipLaunchKernelGGL(k_topk_agg_tiles, dim3(static_cast<unsigned>(nb)), dim3(kBlock), 0, st, w.val, w.idx, D.k, D.M,
                       S.agg_start, S.n_agg_tiles, D.d, D.ld, Qhat, im);
    return hipGetLastError();
}

}  // namespace dq
