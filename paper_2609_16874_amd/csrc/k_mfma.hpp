// k_mfma.hpp -- matrix-core decoder kernels for bin grids up to 32 x 32.
//
// Both passes stream the frame in chunks of 512 pixels per wave: a wave
// reads the foreground channel, compacts the participating pixels with a
// ballot into a per-wave queue in LDS and processes them in tiles of 32.
//
// Per-axis distances (Eq4/Eq10).  S = |X - P|^2 = |X|^2 + |P|^2 - 2 X.P,
// where X.(-2P) is a dense [pixels x channels] x [channels x bins]
// contraction: v_mfma_f32_32x32x16_f16 with X as fp16 (for fp16 inputs every
// clamped, scaled, rounded value is exactly representable; fp32 inputs add
// the residual X - fp16(X) as a second operand) against -2P split into two
// fp16 limbs, -2P = 128 hi + lo with |hi|, |lo| <= 64.  Every partial sum is an integer below 2^24 in
// magnitude, so both fp32 accumulators are exact and S is assembled exactly
// in 32-bit integer arithmetic.
//
// Pass 1, k_vote_mfma (recovery + soft voting, Eq5/Eq6/Eq11).  With pixels
// as the MFMA rows, the distance result leaves in each lane one bin and 16
// pixels -- exactly the operand layout of the vote contraction
// H = Qx^T Qy over pixels, so the weights feed the second MFMA without any
// data exchange between lanes.  A weight q <= 2^15 is split into fp16 limbs
// q = 256 hi + lo; the four limb products accumulate in fp32 exactly as long
// as at most 256 pixels are summed, after which they are folded into 64-bit
// integer sums.
//
// Pass 2, k_assign_mfma (assignment, Eq7, and label write-out).  With the
// palette as MFMA rows each lane holds one pixel and 16 bins; the distance
// codes go through LDS, transposed so that one lane serves one pixel, and
// the candidate search walks the peak rows: the key (c_x + c_y) * 2^14 +
// (128 b + a) is minimised over the peaks, which selects the smallest code
// sum and, on ties, the lowest bin index, i.e. the lowest centroid index.
#pragma once

#include "cpe_common.hpp"

namespace cpe {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

constexpr int kChunk = 512;          // pixels scanned per wave step (8 x 64)
constexpr int kWpb = 4;              // waves per workgroup

template <int F>
struct AxisShape {
    static constexpr int C = 2 * F;             // channels per axis
    static constexpr int KS = (C + 15) / 16;    // MFMA K-steps of 16 channels
};

// Clamp, scale and round a pair of fp16 inputs to fixed-point integers (kept
// as fp16, exact) and accumulate their squares.
__device__ __forceinline__ f16x2 fix_pair_f16(f16x2 v, int32_t &n2)
{
    const f16x2 lo = {(_Float16)-1.5f, (_Float16)-1.5f}, hi = {(_Float16)1.5f, (_Float16)1.5f};
    v = __builtin_elementwise_max(v, lo);
    v = __builtin_elementwise_min(v, hi);
    v = v * (f16x2){(_Float16)4096.0f, (_Float16)4096.0f};
    f16x2 r;
    r[0] = __builtin_rintf16(v[0]);
    r[1] = __builtin_rintf16(v[1]);
    const v2s si = {(short)r[0], (short)r[1]};
    n2 = __builtin_amdgcn_sdot2(si, si, n2, false);
    return r;
}

// fp32 input: X = rint(4096 clamp(v, -1.5, 1.5)) may exceed fp16's 11-bit
// significand, so it is fed to the matrix cores as fp16(X) plus the exact
// residual X - fp16(X) (|residual| <= 2), both accumulated into the same sums.
__device__ __forceinline__ void fix_f32(float v, _Float16 &main, _Float16 &rest, short &si)
{
    const float t = rintf(fminf(fmaxf(v, -1.5f), 1.5f) * 4096.0f);
    si = (short)t;
    main = (_Float16)t;
    rest = (_Float16)(t - (float)main);
}

// Fixed-point channel values of one lane's operand slice.  For fp16 inputs
// every value is exact in fp16 and `rest` stays zero.
struct Fix8 {
    f16x8 main, rest;
};

template <typename T>
constexpr bool kNeedsRest = sizeof(T) == 4;

// Fixed-point values of the 8 channels [16 j + 8 g, 16 j + 8 g + 8) of one
// axis block (channels past 2F read as 0), plus their squares added to n2.
template <typename T, int F>
__device__ __forceinline__ Fix8 load_fix8(const T *__restrict__ blk, int j, int g, int32_t &n2)
{
    constexpr int C = 2 * F;
    const int c0 = 16 * j + 8 * g;
    Fix8 out;
    out.rest = (f16x8){};
    if constexpr (sizeof(T) == 2 && C % 16 == 0) {
        const u32x4 w = *reinterpret_cast<const u32x4 *>(__builtin_assume_aligned(blk + c0, 16));
        const uint32_t words[4] = {w.x, w.y, w.z, w.w};
        u32x4 res;
#pragma unroll
        for (int q = 0; q < 4; q++) {
            const uint32_t word = words[q];
            f16x2 v;
            __builtin_memcpy(&v, &word, 4);
            const f16x2 r = fix_pair_f16(v, n2);
            uint32_t o;
            __builtin_memcpy(&o, &r, 4);
            res[q] = o;
        }
        out.main = __builtin_bit_cast(f16x8, res);
    } else {
        float v[8];
        if constexpr (sizeof(T) == 4 && C % 16 == 0) {
            const float4 *p = reinterpret_cast<const float4 *>(__builtin_assume_aligned(blk + c0, 16));
            const float4 a = p[0], b = p[1];
            v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
            v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
        } else {
#pragma unroll
            for (int s = 0; s < 8; s++) v[s] = (c0 + s) < C ? load_scalar<T>(blk + c0 + s) : 0.0f;
        }
#pragma unroll
        for (int q = 0; q < 4; q++) {
            short s0, s1;
            _Float16 m0, m1, r0, r1;
            fix_f32(v[2 * q], m0, r0, s0);
            fix_f32(v[2 * q + 1], m1, r1, s1);
            out.main[2 * q] = m0;
            out.main[2 * q + 1] = m1;
            out.rest[2 * q] = r0;
            out.rest[2 * q + 1] = r1;
            const v2s si = {s0, s1};
            n2 = __builtin_amdgcn_sdot2(si, si, n2, false);
        }
    }
    return out;
}

// Palette operand of lane (bin = lane & 31, group g) for K-step j: the limb
// of -2P at channels [16 j + 8 g, +8), from the [32 bins][32 channels] table.
__device__ __forceinline__ f16x8 palette_operand(const int8_t *__restrict__ limb, int bin, int j, int g)
{
    f16x8 out;
#pragma unroll
    for (int s = 0; s < 8; s++) out[s] = (_Float16)(float)limb[bin * 32 + 16 * j + 8 * g + s];
    return out;
}

// Row of the 32 x 32 MFMA result held by register r of a lane in group g.
__device__ __forceinline__ constexpr int acc_row(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }

__device__ __forceinline__ f32x16 mfma16(f16x8 a, f16x8 b, f32x16 c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// Pass 1: recovery + soft voting
// ---------------------------------------------------------------------------
template <typename T, int F>
__global__ __launch_bounds__(256) void k_vote_mfma(const T *__restrict__ emb, const T *__restrict__ fg, int32_t npix,
                                                   float fg_thr, Tables tb, int32_t Bw, int32_t Bh,
                                                   unsigned long long *__restrict__ hrep)
{
    constexpr int KS = AxisShape<F>::KS;
    constexpr int D = 4 * F;
    extern __shared__ __align__(16) unsigned char smem[];
    uint32_t *s_wt = reinterpret_cast<uint32_t *>(smem);                              // [kWKeys]
    unsigned long long *s_h = reinterpret_cast<unsigned long long *>(s_wt + kWKeys);  // [32 * 32]
    int32_t *s_q = reinterpret_cast<int32_t *>(s_h + kMfmaBins * kMfmaBins);         // [kWpb][96]
    int32_t *s_nrm = s_q + kWpb * 96;                                                 // [kWpb][64]

    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int g = lane >> 5, ln = lane & 31;
    for (int i = tid; i < kWKeys; i += blockDim.x) s_wt[i] = tb.wt_pk[i];
    for (int i = tid; i < kMfmaBins * kMfmaBins; i += blockDim.x) s_h[i] = 0ull;
    __syncthreads();

    f16x8 pxh[KS], pxl[KS], pyh[KS], pyl[KS];
#pragma unroll
    for (int j = 0; j < KS; j++) {
        pxh[j] = palette_operand(tb.qx, ln, j, g);
        pxl[j] = palette_operand(tb.qx + 1024, ln, j, g);
        pyh[j] = palette_operand(tb.qy, ln, j, g);
        pyl[j] = palette_operand(tb.qy + 1024, ln, j, g);
    }
    const uint32_t np1x = tb.np1_x[ln], np1y = tb.np1_y[ln];

    int32_t *q = s_q + wv * 96;
    int32_t *nrm = s_nrm + wv * 64;
    f32x16 acc2 = {}, acc1 = {}, acc0 = {};
    unsigned long long H[16];
#pragma unroll
    for (int r = 0; r < 16; r++) H[r] = 0ull;
    int ntile = 0;

    auto fold = [&]() {
#pragma unroll
        for (int r = 0; r < 16; r++) {
            H[r] += ((unsigned long long)(uint32_t)acc2[r] << 16) + ((unsigned long long)(uint32_t)acc1[r] << 8) +
                    (unsigned long long)(uint32_t)acc0[r];
            acc2[r] = 0.0f;
            acc1[r] = 0.0f;
            acc0[r] = 0.0f;
        }
    };

    // One tile of up to 32 queued pixels: slot m = lane & 31 of the tile.
    auto tile = [&](int nvalid) {
        const int pix = q[ln < nvalid ? ln : 0];
        const T *row = emb + (size_t)pix * D;
        int32_t n2x = 0, n2y = 0;
        Fix8 X[KS], Y[KS];
#pragma unroll
        for (int j = 0; j < KS; j++) {
            X[j] = load_fix8<T, F>(row, j, g, n2x);
            Y[j] = load_fix8<T, F>(row + 2 * F, j, g, n2y);
        }
        n2x += __shfl_xor(n2x, 32);
        n2y += __shfl_xor(n2y, 32);
        if (g == 0) {
            nrm[ln] = n2x;
            nrm[32 + ln] = n2y;
        }
        f32x16 ah = {}, al = {};
#pragma unroll
        for (int j = 0; j < KS; j++) {
            ah = mfma16(X[j].main, pxh[j], ah);
            al = mfma16(X[j].main, pxl[j], al);
            if constexpr (kNeedsRest<T>) {
                ah = mfma16(X[j].rest, pxh[j], ah);
                al = mfma16(X[j].rest, pxl[j], al);
            }
        }
        uint32_t ex[16], ey[16];
#pragma unroll
        for (int r4 = 0; r4 < 4; r4++) {
            const i32x4 n4 = *reinterpret_cast<const i32x4 *>(nrm + 8 * r4 + 4 * g);
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int r = 4 * r4 + i;
                const uint32_t s1 = (uint32_t)((int32_t)ah[r] * 128 + (int32_t)al[r]) + (uint32_t)n4[i] + np1x;
                const uint32_t bits = __float_as_uint((float)s1);
                ex[r] = s_wt[(bits >> 15) & (kWKeys - 1)];
            }
        }
        if (nvalid < 32) {
#pragma unroll
            for (int r = 0; r < 16; r++)
                if (acc_row(r, g) >= nvalid) ex[r] = 0u;
        }
        ah = (f32x16){};
        al = (f32x16){};
#pragma unroll
        for (int j = 0; j < KS; j++) {
            ah = mfma16(Y[j].main, pyh[j], ah);
            al = mfma16(Y[j].main, pyl[j], al);
            if constexpr (kNeedsRest<T>) {
                ah = mfma16(Y[j].rest, pyh[j], ah);
                al = mfma16(Y[j].rest, pyl[j], al);
            }
        }
#pragma unroll
        for (int r4 = 0; r4 < 4; r4++) {
            const i32x4 n4 = *reinterpret_cast<const i32x4 *>(nrm + 32 + 8 * r4 + 4 * g);
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int r = 4 * r4 + i;
                const uint32_t s1 = (uint32_t)((int32_t)ah[r] * 128 + (int32_t)al[r]) + (uint32_t)n4[i] + np1y;
                const uint32_t bits = __float_as_uint((float)s1);
                ey[r] = s_wt[(bits >> 15) & (kWKeys - 1)];
            }
        }
        // vote: K = the 16 pixels of this lane, in two MFMAs of 8
#pragma unroll
        for (int t = 0; t < 2; t++) {
            u32x4 xl, xh, yl, yh;
#pragma unroll
            for (int s = 0; s < 4; s++) {
                const int r = 8 * t + 2 * s;
                xl[s] = __builtin_amdgcn_perm(ex[r + 1], ex[r], 0x05040100u);
                xh[s] = __builtin_amdgcn_perm(ex[r + 1], ex[r], 0x07060302u);
                yl[s] = __builtin_amdgcn_perm(ey[r + 1], ey[r], 0x05040100u);
                yh[s] = __builtin_amdgcn_perm(ey[r + 1], ey[r], 0x07060302u);
            }
            const f16x8 XL = __builtin_bit_cast(f16x8, xl), XH = __builtin_bit_cast(f16x8, xh);
            const f16x8 YL = __builtin_bit_cast(f16x8, yl), YH = __builtin_bit_cast(f16x8, yh);
            acc2 = mfma16(XH, YH, acc2);
            acc1 = mfma16(XH, YL, acc1);
            acc1 = mfma16(XL, YH, acc1);
            acc0 = mfma16(XL, YL, acc0);
        }
        if (++ntile == 8) {        // 256 pixels: fold before an fp32 sum could exceed 2^24
            fold();
            ntile = 0;
        }
    };

    const int nchunks = (int)(((int64_t)npix + kChunk - 1) / kChunk);
    const int nw = gridDim.x * kWpb;
    int qn = 0;
    for (int c = blockIdx.x * kWpb + wv; c < nchunks; c += nw) {
        const int base = c * kChunk;
        float fv[8];
#pragma unroll
        for (int i = 0; i < 8; i++) {
            const int p = base + 64 * i + lane;
            fv[i] = p < npix ? load_scalar<T>(fg + p) : 0.0f;
        }
#pragma unroll
        for (int i = 0; i < 8; i++) {
            const int p = base + 64 * i + lane;
            const bool f = p < npix && fv[i] > fg_thr;
            const unsigned long long m = __ballot(f);
            if (f) q[qn + lane_prefix(m)] = p;
            qn += __popcll(m);
            while (qn >= 32) {
                tile(32);
                qn -= 32;
                const int moved = lane < qn ? q[32 + lane] : 0;
                if (lane < qn) q[lane] = moved;
            }
        }
    }
    if (qn > 0) tile(qn);
    fold();

    // block reduction of the 32 x 32 histogram, then one atomic per bin
#pragma unroll
    for (int r = 0; r < 16; r++) {
        const int a = acc_row(r, g), b = ln;
        if (a < Bw && b < Bh && H[r]) atomicAdd(&s_h[b * kMfmaBins + a], H[r]);
    }
    __syncthreads();
    const int nb = Bw * Bh;
    unsigned long long *dst = hrep + (size_t)(blockIdx.x % kReplicas) * nb;
    for (int i = tid; i < kMfmaBins * kMfmaBins; i += blockDim.x) {
        const int b = i / kMfmaBins, a = i % kMfmaBins;
        if (a < Bw && b < Bh && s_h[i]) atomicAdd(dst + b * Bw + a, s_h[i]);
    }
}

// ---------------------------------------------------------------------------
// Pass 2: assignment + label write-out
// ---------------------------------------------------------------------------
constexpr int kWpb2 = 8;             // waves per workgroup of the assignment kernel

// LDS bytes of k_assign_mfma: code table, bin -> centroid table, counts,
// row masks, and per wave a queue, x keys [32 bins][64 lanes] (u32) and
// y codes [32 bins][64 lanes] (u16).
constexpr size_t kAssignLds = (size_t)kCKeys * 2 + kMfmaBins * kMfmaBins * 2 + kMfmaBins * kMfmaBins * 4 +
                              kMfmaBins * 4 + (size_t)kWpb2 * (128 * 4 + kMfmaBins * 64 * 4 + kMfmaBins * 64 * 2);

template <typename T, int F>
__global__ __launch_bounds__(512) void k_assign_mfma(const T *__restrict__ emb, const T *__restrict__ fg,
                                                     int32_t npix, float fg_thr, Tables tb,
                                                     const uint32_t *__restrict__ rowmask,
                                                     const uint16_t *__restrict__ rank,
                                                     const int32_t *__restrict__ kinfo,
                                                     cpe_centroid *__restrict__ cents, int32_t *__restrict__ labels,
                                                     float *__restrict__ score_map)
{
    constexpr int KS = AxisShape<F>::KS;
    constexpr int D = 4 * F;
    extern __shared__ __align__(16) unsigned char smem[];
    uint16_t *s_ct = reinterpret_cast<uint16_t *>(smem);                          // [kCKeys]
    uint16_t *s_rank = s_ct + kCKeys;                                              // [32 * 32]
    int32_t *s_cnt = reinterpret_cast<int32_t *>(s_rank + kMfmaBins * kMfmaBins);  // [1024]
    uint32_t *s_rm = reinterpret_cast<uint32_t *>(s_cnt + kMfmaBins * kMfmaBins); // [32]
    int32_t *s_q = reinterpret_cast<int32_t *>(s_rm + kMfmaBins);                 // [kWpb2][128]
    uint32_t *s_kx = reinterpret_cast<uint32_t *>(s_q + kWpb2 * 128);             // [kWpb2][32][64]
    uint16_t *s_cy = reinterpret_cast<uint16_t *>(s_kx + kWpb2 * kMfmaBins * 64); // [kWpb2][32][64]

    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int g = lane >> 5, ln = lane & 31;
    const int Kc = kinfo[0];
    const int nchunks = (int)(((int64_t)npix + kChunk - 1) / kChunk);
    const int nw = gridDim.x * kWpb2;

    if (Kc == 0) {              // no centroid: every pixel is unlabelled
        for (int c = blockIdx.x * kWpb2 + wv; c < nchunks; c += nw)
#pragma unroll
            for (int i = 0; i < 8; i++) {
                const int p = c * kChunk + 64 * i + lane;
                if (p < npix) {
                    labels[p] = 0;
                    if (score_map) score_map[p] = 0.0f;
                }
            }
        return;
    }

    for (int i = tid; i < kCKeys; i += blockDim.x) s_ct[i] = tb.ct_pm[i];
    for (int i = tid; i < kMfmaBins * kMfmaBins; i += blockDim.x) {
        s_rank[i] = rank[i];
        s_cnt[i] = 0;
    }
    if (tid < kMfmaBins) s_rm[tid] = rowmask[tid];
    __syncthreads();

    f16x8 pxh[KS], pxl[KS], pyh[KS], pyl[KS];
#pragma unroll
    for (int j = 0; j < KS; j++) {
        pxh[j] = palette_operand(tb.qx, ln, j, g);
        pxl[j] = palette_operand(tb.qx + 1024, ln, j, g);
        pyh[j] = palette_operand(tb.qy, ln, j, g);
        pyl[j] = palette_operand(tb.qy + 1024, ln, j, g);
    }
    uint32_t npx[16], npy[16];
#pragma unroll
    for (int r = 0; r < 16; r++) {
        npx[r] = tb.np1_x[acc_row(r, g)];
        npy[r] = tb.np1_y[acc_row(r, g)];
    }

    int32_t *q = s_q + wv * 128;
    uint32_t *kx = s_kx + wv * kMfmaBins * 64;     // x key of bin a, pixel slot p: kx[a * 64 + p]
    uint16_t *cyb = s_cy + wv * kMfmaBins * 64;    // y code of bin b, pixel slot p: cyb[b * 64 + p]

    // Keys of one tile of 32 pixels (queue slots 32 t .. 32 t + 31).
    auto codes = [&](int t, int nvalid) {
        const int slot = 32 * t + ln;
        const int pix = q[slot < nvalid ? slot : 0];
        const T *row = emb + (size_t)pix * D;
        int32_t n2x = 0, n2y = 0;
        Fix8 X[KS], Y[KS];
#pragma unroll
        for (int j = 0; j < KS; j++) {
            X[j] = load_fix8<T, F>(row, j, g, n2x);
            Y[j] = load_fix8<T, F>(row + 2 * F, j, g, n2y);
        }
        n2x += __shfl_xor(n2x, 32);
        n2y += __shfl_xor(n2y, 32);
        f32x16 ah = {}, al = {};
#pragma unroll
        for (int j = 0; j < KS; j++) {
            ah = mfma16(pxh[j], X[j].main, ah);
            al = mfma16(pxl[j], X[j].main, al);
            if constexpr (kNeedsRest<T>) {
                ah = mfma16(pxh[j], X[j].rest, ah);
                al = mfma16(pxl[j], X[j].rest, al);
            }
        }
#pragma unroll
        for (int r = 0; r < 16; r++) {
            const uint32_t s1 = (uint32_t)((int32_t)ah[r] * 128 + (int32_t)al[r]) + (uint32_t)n2x + npx[r];
            const uint32_t bits = __float_as_uint((float)s1);
            const uint32_t code = s_ct[(bits >> 14) & (kCKeys - 1)];
            const int a = acc_row(r, g);
            kx[a * 64 + slot] = (code << 14) | (uint32_t)a;
        }
        ah = (f32x16){};
        al = (f32x16){};
#pragma unroll
        for (int j = 0; j < KS; j++) {
            ah = mfma16(pyh[j], Y[j].main, ah);
            al = mfma16(pyl[j], Y[j].main, al);
            if constexpr (kNeedsRest<T>) {
                ah = mfma16(pyh[j], Y[j].rest, ah);
                al = mfma16(pyl[j], Y[j].rest, al);
            }
        }
#pragma unroll
        for (int r = 0; r < 16; r++) {
            const uint32_t s1 = (uint32_t)((int32_t)ah[r] * 128 + (int32_t)al[r]) + (uint32_t)n2y + npy[r];
            const uint32_t bits = __float_as_uint((float)s1);
            cyb[acc_row(r, g) * 64 + slot] = s_ct[(bits >> 14) & (kCKeys - 1)];
        }
    };

    // Candidate search for up to 64 queued pixels (lane p: queue slot p):
    // per peak row b, m = min over its peak columns a of x key, then
    // best = min(best, m + y key of b).
    auto group = [&](int nvalid) {
        codes(0, nvalid);
        if (nvalid > 32) codes(1, nvalid);
        const uint32_t *kxl = kx + lane;
        uint32_t best = 0xffffffffu;
#pragma unroll
        for (int b = 0; b < kMfmaBins; b++) {
            uint32_t mb = __builtin_amdgcn_readfirstlane(s_rm[b]);
            if (mb) {
                const uint32_t ky = ((uint32_t)cyb[b * 64 + lane] << 14) | ((uint32_t)b << 7);
                uint32_t m = 0xffffffffu;
                while (mb) {
                    const int a = __builtin_ctz(mb);
                    mb &= mb - 1u;
                    m = min(m, kxl[a * 64]);
                }
                best = min(best, m + ky);
            }
        }
        if (lane < nvalid) {
            const int pix = q[lane];
            // a, b < 32 here (the row masks only hold bins of the grid); the
            // masks keep the table reads in bounds regardless
            const int a = (int)(best & 31u), b = (int)((best >> 7) & 31u);
            const int k = s_rank[b * kMfmaBins + a] & (kMfmaBins * kMfmaBins - 1);
            labels[pix] = k + 1;
            if (score_map) score_map[pix] = expf(-((float)(best >> 14) * 0x1p-12f));
            atomicAdd(s_cnt + k, 1);
        }
    };

    int qn = 0;
    for (int c = blockIdx.x * kWpb2 + wv; c < nchunks; c += nw) {
        const int base = c * kChunk;
        float fv[8];
#pragma unroll
        for (int i = 0; i < 8; i++) {
            const int p = base + 64 * i + lane;
            fv[i] = p < npix ? load_scalar<T>(fg + p) : 0.0f;
        }
#pragma unroll
        for (int i = 0; i < 8; i++) {
            const int p = base + 64 * i + lane;
            const bool f = p < npix && fv[i] > fg_thr;
            if (p < npix && !f) {
                labels[p] = 0;
                if (score_map) score_map[p] = 0.0f;
            }
            const unsigned long long m = __ballot(f);
            if (f) q[qn + lane_prefix(m)] = p;
            qn += __popcll(m);
            if (qn >= 64) {
                group(64);
                qn -= 64;
                const int moved = lane < qn ? q[64 + lane] : 0;
                if (lane < qn) q[lane] = moved;
            }
        }
    }
    if (qn > 0) group(qn);
    __syncthreads();
    for (int i = tid; i < Kc && i < kMfmaBins * kMfmaBins; i += blockDim.x)
        if (s_cnt[i]) atomicAdd(&cents[i].npix, s_cnt[i]);
}

}  // namespace cpe
