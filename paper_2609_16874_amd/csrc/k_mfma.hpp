// k_mfma.hpp -- matrix-core decoder kernels for bin grids up to 32 x 32.
//
// Both passes stream the compact list of participating pixels written by
// k_compact (or every pixel, when the frame has no foreground channel): the
// list is cut into tiles of 32 consecutive entries, every workgroup gets a
// contiguous run of tiles of the same length to within one, and its waves
// take the run's tiles one at a time from a counter in LDS (so that they
// finish together however the SIMDs favour older waves), always loading the
// embedding rows of the next tile (and the list entries of the one after)
// before computing the current one.  Every tile but the last is full.
//
// Per-axis distances (Eq4/Eq10).  With the input on its 1/256 grid,
// X = 16 Xr (Xr = rint(256 clamp(v, -1.5, 1.5)), |Xr| <= 384, exact in fp16)
// and the palette limbs -2P = 128 hi + lo (|hi|, |lo| <= 64, exact in fp16),
// S + 1 = 256 |Xr|^2 + (|P|^2 + 1) + 16 (128 Xr.hi + Xr.lo).  The two dot
// products are dense [pixels x channels] x [channels x bins] contractions:
// v_mfma_f32_32x32x16_f16 accumulating onto 1.5 * 2^23, where every partial
// sum (at most 32 * 384 * 64 < 2^22 in magnitude) stays in the binade of unit
// spacing, so the accumulator's bit pattern minus 0x4B400000 is the exact
// integer: S + 1 follows from the two bit patterns with two shift-adds and
// one add, modulo 2^32 (S + 1 < 2^32).  |Xr|^2 <= 32 * 384^2 < 2^24 is an
// exact fp32 dot product of the fp16 operands.
//
// Pass 1, k_vote_mfma (recovery + soft voting, Eq5/Eq6/Eq11).  With pixels
// as the MFMA rows, the distance result leaves in each lane one bin and 16
// pixels -- exactly the operand layout of the vote contraction
// H = Qx^T Qy over pixels, so the weights feed the second MFMA without any
// data exchange between lanes.  A weight q <= 2^15 is split into fp16 limbs
// q = 256 hi + lo; the four limb products accumulate in fp32 exactly as long
// as at most 256 pixels are summed, after which they are added into a 64-bit
// histogram in LDS.
//
// Pass 2, k_assign_mfma (assignment, Eq7, and label write-out).  Only the
// candidate columns and rows are needed: they are numbered in ascending
// order (slots), the MFMA rows are the slots' palette entries, each lane
// holds one pixel and 16 slots, and codes are computed for the groups of 8
// slots that hold candidates.  The codes go to LDS as the high halves of
// search keys whose low halves hold the slot index, laid out so that one lane
// serves one pixel, and the candidate search walks the batches of 4 columns
// of one row: the key (c_x + c_y) * 2^16 + (128 row slot + column slot) is
// minimised over the peaks, which selects the smallest code sum and, on
// ties, the lowest (row, column) -- slots keep the bins' order -- i.e. the
// lowest centroid index.
#pragma once

#include "cpe_common.hpp"
#include "k_compact.hpp"
#include "k_peaks.hpp"

namespace cpe {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

constexpr int kWpb2 = 12;            // waves per workgroup of the assignment kernel (3 per SIMD)
constexpr int kPopBytes = 2 * 2 * 2 * 64 * 16;   // palette operands of both axes, limbs and K-steps

template <int F>
struct AxisShape {
    static constexpr int C = 2 * F;             // channels per axis
    static constexpr int KS = (C + 15) / 16;    // MFMA K-steps of 16 channels
};

// The fp32 value 1.5 * 2^23 (bit pattern 0x4B400000) onto which the limb
// accumulators are summed.
constexpr float kMagic = 12582912.0f;
constexpr uint32_t kMagicBits = 0x4B400000u;

// Round a pair of fp16 inputs to the 1/256 grid, clamped to [-1.5, 1.5]:
// Xr = rint(256 v) as fp16, and accumulate Xr^2 (exact in fp32).  The
// rounding is one fused multiply-add onto 1536: for |256 v| <= 512 the sum
// lies in [1024, 2048], where fp16 spacing is 1, so it is rounded to the
// nearest integer, ties to even (1536 is even); larger magnitudes (and
// overflow to +-inf) leave that range and are clamped to 1536 +- 384 like
// any value beyond 1.5.  A NaN clamps to 1536 - 384 (max returns the
// non-NaN operand), i.e. to -1.5.
__device__ __forceinline__ f16x2 fix_pair_f16(f16x2 v, float &n2)
{
    const f16x2 k256 = {(_Float16)256.0f, (_Float16)256.0f}, k1536 = {(_Float16)1536.0f, (_Float16)1536.0f};
    const f16x2 lo = {(_Float16)1152.0f, (_Float16)1152.0f}, hi = {(_Float16)1920.0f, (_Float16)1920.0f};
    f16x2 r = __builtin_elementwise_fma(v, k256, k1536);
    r = __builtin_elementwise_max(r, lo);
    r = __builtin_elementwise_min(r, hi);
    r = r - k1536;
    n2 = __builtin_amdgcn_fdot2(r, r, n2, false);
    return r;
}

// fp32 input: Xr = rint(256 clamp(v, -1.5, 1.5)) (a NaN clamps to -1.5, as
// fmaxf returns the non-NaN operand), exact in fp16.
__device__ __forceinline__ _Float16 fix_f32(float v)
{
    return (_Float16)rintf(fminf(fmaxf(v * 256.0f, -384.0f), 384.0f));
}

// Raw input words of one lane's operand slices: for each axis and K-step j
// the 8 channels [16 j + 8 g, 16 j + 8 g + 8) of one pixel's axis block
// (channels past 2F read as 0).  Loaded one tile ahead of their use.
template <typename T, int F>
struct RawSlices {
    static constexpr int C = 2 * F;
    static constexpr int KS = AxisShape<F>::KS;
    static constexpr bool kH = sizeof(T) == 2;
    // 16-byte aligned vector slices: whole K-steps, or a single 8-channel
    // slice per axis (F = 4) that the lanes of half 0 load
    static constexpr bool kVec = C % 16 == 0 || C == 8;
    static constexpr int kWords = (kH && kVec) ? 4 : 8;
    uint32_t w[2][KS][kWords];

    // `row` = first channel of the pixel, `yoff` = first channel of its y
    // block.  The host guarantees that every vector slice is 16-byte aligned
    // (16-byte aligned embedding; 2F a multiple of 16, or 2F = 8 with the
    // row and the y block 16-byte aligned).
    __device__ __forceinline__ void load(const T *__restrict__ row, int yoff, int g)
    {
#pragma unroll
        for (int ax = 0; ax < 2; ax++)
#pragma unroll
            for (int j = 0; j < KS; j++) {
                const T *blk = row + ax * yoff + 16 * j + 8 * g;
                if constexpr (kVec) {
                    // C == 8: the slice of half 1 lies past the block; it reads
                    // the half-0 slice (in bounds) and keeps zeros
                    const bool on = C % 16 == 0 || g == 0;
                    const T *src = on ? blk : row + ax * yoff + 16 * j;
                    if constexpr (kH) {
                        const u32x4 v = *reinterpret_cast<const u32x4 *>(__builtin_assume_aligned(src, 16));
#pragma unroll
                        for (int q = 0; q < 4; q++) w[ax][j][q] = on ? v[q] : 0u;
                    } else {
                        const float4 *p = reinterpret_cast<const float4 *>(__builtin_assume_aligned(src, 16));
                        const float4 a = p[0], b = p[1];
                        const float f[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
                        for (int q = 0; q < 8; q++) w[ax][j][q] = on ? __float_as_uint(f[q]) : 0u;
                    }
                } else {
#pragma unroll
                    for (int s = 0; s < 8; s++)
                        w[ax][j][s] =
                            __float_as_uint((16 * j + 8 * g + s) < C ? load_scalar<T>(blk + s) : 0.0f);
                }
            }
    }

    // Rounded operands of one axis and its partial |Xr|^2.
    __device__ __forceinline__ void convert(int ax, f16x8 (&X)[KS], float &n2) const
    {
#pragma unroll
        for (int j = 0; j < KS; j++) {
            if constexpr (kH && kVec) {
                u32x4 res;
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    const uint32_t word = w[ax][j][q];
                    f16x2 v;
                    __builtin_memcpy(&v, &word, 4);
                    const f16x2 r = fix_pair_f16(v, n2);
                    uint32_t o;
                    __builtin_memcpy(&o, &r, 4);
                    res[q] = o;
                }
                X[j] = __builtin_bit_cast(f16x8, res);
            } else {
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    const f16x2 r = {fix_f32(__uint_as_float(w[ax][j][2 * q])),
                                     fix_f32(__uint_as_float(w[ax][j][2 * q + 1]))};
                    X[j][2 * q] = r[0];
                    X[j][2 * q + 1] = r[1];
                    n2 = __builtin_amdgcn_fdot2(r, r, n2, false);
                }
            }
        }
    }
};

// Palette operand of lane `lane` (bin lane & 31, channels 16 j + 8 (lane >> 5)
// + 0..7) for axis ax (0 = x, 1 = y), limb (0 = hi, 1 = lo) and K-step j.
__device__ __forceinline__ f16x8 palette_operand(const uint32_t *__restrict__ pop, int ax, int limb, int j, int lane)
{
    const u32x4 w = *reinterpret_cast<const u32x4 *>(pop + ((((ax * 2 + limb) * 2 + j) * 64 + lane) * 4));
    return __builtin_bit_cast(f16x8, w);
}

// Row of the 32 x 32 MFMA result held by register r of a lane in group g.
__device__ __forceinline__ constexpr int acc_row(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }

__device__ __forceinline__ f32x16 mfma16(f16x8 a, f16x8 b, f32x16 c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// Xr.hi and Xr.lo of one axis, accumulated onto the starting values ah, al
// (kMagic plus the pixel's part, see below).
// PIX_ROWS: pixels are the MFMA rows (pass 1) or its columns (pass 2).
template <int KS, bool PIX_ROWS>
__device__ __forceinline__ void axis_dot(const f16x8 (&X)[KS], const f16x8 (&ph)[KS], const f16x8 (&pl)[KS],
                                         f32x16 &ah, f32x16 &al)
{
#pragma unroll
    for (int j = 0; j < KS; j++) {
        if constexpr (PIX_ROWS) {
            ah = mfma16(X[j], ph[j], ah);
            al = mfma16(X[j], pl[j], al);
        } else {
            ah = mfma16(ph[j], X[j], ah);
            al = mfma16(pl[j], X[j], al);
        }
    }
}

// S + 1 = 2048 A + 16 L + 256 |Xr|^2 + |P|^2 + 1 with A = Xr.hi and L =
// Xr.lo.  The pixel's part 256 |Xr|^2 = 2048 (|Xr|^2 >> 3) + 16 (16 (|Xr|^2
// & 7)) starts the two accumulators: ah = kMagic + (|Xr|^2 >> 3) + A and
// al = kMagic + 16 (|Xr|^2 & 7) + L, both integers within 2^22 of kMagic,
// so exact in fp32 and bits(ah) = 0x4B400000 + their offset.  Then
// S + 1 = 2048 bits(ah) + 16 bits(al) + c (mod 2^32) with the bin's
// constant c = |P|^2 + 1 - 2064 * 0x4B400000, and S + 1 < 2^32.
struct PixelInit {
    uint32_t a, l;    // bit patterns of the starting values of ah and al
};
__device__ __forceinline__ PixelInit pixel_init(float n2)
{
    const uint32_t u = (uint32_t)n2;    // |Xr|^2 <= 32 * 384^2, exact in fp32
    return {kMagicBits + (u >> 3), kMagicBits + ((u & 7u) << 4)};
}
__device__ __forceinline__ uint32_t bin_const(uint32_t np1) { return np1 - 2064u * kMagicBits; }

// Bits of fl32(S + 1) from the two accumulators and the remaining constant
// (the bin's constant, plus 256 |Xr|^2 when both accumulators start at
// kMagic), as
// two shift-and-add instructions: the empty asm makes the first sum opaque,
// which keeps the compiler from forming two shifts and a three-way add.
// (The instructions themselves stay compiler-generated: the accumulators
// are MFMA results, and only the compiler inserts the wait states a read of
// them needs.)
__device__ __forceinline__ uint32_t s1_bits(float ah, float al, uint32_t c)
{
    uint32_t t = (__float_as_uint(al) << 4) + c;
    asm("" : "+v"(t));
    return __float_as_uint((float)((__float_as_uint(ah) << 11) + t));
}

// Starting values of one accumulator for the 16 pixels (rows acc_row(r, g))
// of a lane in group g, from a per-wave LDS array indexed by pixel.
__device__ __forceinline__ f32x16 row_init(const uint32_t *a, int g)
{
    f32x16 v;
#pragma unroll
    for (int r4 = 0; r4 < 4; r4++) {
        const u32x4 w = *reinterpret_cast<const u32x4 *>(a + 8 * r4 + 4 * g);
#pragma unroll
        for (int i = 0; i < 4; i++) v[4 * r4 + i] = __uint_as_float(w[i]);
    }
    return v;
}

// Tiles [first, last) of workgroup b of nb when ntiles tiles are shared out
// in contiguous runs.
__device__ __forceinline__ void block_run(int ntiles, int b, int nb, int &first, int &last)
{
    first = (int)((int64_t)ntiles * b / nb);
    last = (int)((int64_t)ntiles * (b + 1) / nb);
}

// Tiles of a workgroup's run: wave w starts with tile first + w, later
// tiles come from an LDS counter (zeroed before the run) in taking order,
// tile first + waves + k for the k-th taker (wave-uniform).
__device__ __forceinline__ int take_tile(int *next, int lane, int first, int waves)
{
    int k = 0;
    if (lane == 0) k = atomicAdd(next, 1);
    return first + waves + __builtin_amdgcn_readfirstlane(k);
}

// ---------------------------------------------------------------------------
// Pass 1: recovery + soft voting (+ the peak extraction in the last workgroup)
// ---------------------------------------------------------------------------
// Row stride (in 64-bit words) of the vote kernel's LDS histogram: one word
// of padding per row puts the 32 rows that one fold instruction touches
// (lanes = y bins, fixed x bin) into distinct banks.
constexpr int kHStride = kMfmaBins + 1;

// LDS bytes of k_vote_mfma: the packed weight table, the 64-bit histogram,
// the palette operands, and per wave the accumulator starting values of one
// tile's pixels.
constexpr size_t kVoteLds(int wpb)
{
    return (size_t)kWKeys * 4 + kMfmaBins * kHStride * 8 + kPopBytes + (size_t)wpb * 128 * 4 + (kMaxSlices + 1) * 4 +
           16;
}

// Waves per SIMD the register allocation must allow: three for fp16 inputs
// with up to 8 or exactly 16 harmonics (one workgroup of 12 waves per compute
// unit), two otherwise (fp32 residual operands, scalar channel loads),
// where three would spill.  Without a bound the compiler keeps the
// accumulators in a separate AGPR allocation and the kernel drops to one wave
// per SIMD.
template <typename T, int F>
constexpr int kVoteWaves = (sizeof(T) == 2 && (F <= 8 || F == 16)) ? 3 : 2;
// Waves per workgroup of the vote kernel: one workgroup per compute unit.
template <typename T, int F>
constexpr int kVoteWpb = 4 * kVoteWaves<T, F>;
//
// Every workgroup adds its histogram into one of the kReplicas vote
// histograms `hrep` (zeroed beforehand); the assignment launch that follows
// sums them and extracts the peaks.  Workgroup 0 also resets the pixel
// counts of the centroid records, which the assignment launch accumulates.
template <typename T, int F>
__global__ __launch_bounds__((kVoteWpb<T, F> * 64)) __attribute__((amdgpu_waves_per_eu(kVoteWaves<T, F>))) void k_vote_mfma(
    const T *__restrict__ emb, int32_t dstride, int32_t yoff, const int32_t *__restrict__ list,
    const int32_t *__restrict__ counts, int32_t nslices, int32_t slice_px, int32_t npix, Tables tb, int32_t Bw,
    int32_t Bh, unsigned long long *__restrict__ hrep,
    cpe_centroid *__restrict__ cents, int32_t cap)
{
    constexpr int KS = AxisShape<F>::KS;
    constexpr int kWpb = kVoteWpb<T, F>;
    // All LDS is static, so that table addresses are compile-time constants.
    __shared__ __align__(16) unsigned char smem[kVoteLds(kWpb)];
    uint32_t *s_wt = reinterpret_cast<uint32_t *>(smem);                              // [kWKeys] fp16 limb pairs
    unsigned long long *s_h = reinterpret_cast<unsigned long long *>(s_wt + kWKeys);  // [32][kHStride], b * kHStride + a
    uint32_t *s_pop = reinterpret_cast<uint32_t *>(s_h + kMfmaBins * kHStride);      // palette operands
    uint32_t *s_ini = s_pop + kPopBytes / 4;                                          // [kWpb][4][32]
    int *s_pref = reinterpret_cast<int *>(s_ini + kWpb * 128);                       // [kMaxSlices + 1]
    int *s_next = s_pref + kMaxSlices + 1;                                            // next tile of the run

    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int g = lane >> 5, ln = lane & 31;
    SliceLoad sl;
    if (list) slice_load(counts, nslices, sl);
    // the bin constants of this lane's bin (loaded with the tables, not after
    // the barrier, where they would cost a memory round trip of their own)
    const uint32_t np1x = tb.np1_x[ln], np1y = tb.np1_y[ln];
    {
        constexpr int kThreads = kWpb * 64, kN = kWKeys / 4, kPer = (kN + kThreads - 1) / kThreads;
        u32x4 w[kPer];
#pragma unroll
        for (int k = 0; k < kPer; k++) {
            const int i = k * kThreads + tid;
            w[k] = reinterpret_cast<const u32x4 *>(tb.wt_pk)[i < kN ? i : 0];
        }
#pragma unroll
        for (int k = 0; k < kPer; k++) {
            const int i = k * kThreads + tid;
            if (i < kN) reinterpret_cast<u32x4 *>(s_wt)[i] = w[k];
        }
        for (int i = tid; i < kMfmaBins * kHStride; i += kThreads) s_h[i] = 0ull;
        for (int i = tid; i < kPopBytes / 16; i += kThreads)
            reinterpret_cast<u32x4 *>(s_pop)[i] = reinterpret_cast<const u32x4 *>(tb.pop)[i];
        if (tid == 0) *s_next = 0;
        if (list) slice_scan(sl, nslices, s_pref);
    }
    __syncthreads();
    // the workgroup's run of tiles
    const int n = list ? s_pref[nslices] : npix, ntiles = (n + 31) >> 5;
    int t0, tend;
    block_run(ntiles, blockIdx.x, gridDim.x, t0, tend);
    const uint32_t cbx = bin_const(np1x), cby = bin_const(np1y);

    // this wave's starting values: [0] x ah, [1] x al, [2] y ah, [3] y al, by pixel
    uint32_t *ini = s_ini + wv * 128;
    f32x16 acc2 = {}, acc1 = {}, acc0 = {};
    int ntile = 0;

    // Add the limb sums into the workgroup's histogram (this wave owns every
    // (a, b) exactly once, so its own atomics never collide).
    auto fold = [&]() {
#pragma unroll
        for (int r = 0; r < 16; r++) {
            const unsigned long long v = ((unsigned long long)(uint32_t)acc2[r] << 16) +
                                         ((unsigned long long)(uint32_t)acc1[r] << 8) +
                                         (unsigned long long)(uint32_t)acc0[r];
            atomicAdd(&s_h[ln * kHStride + acc_row(r, g)], v);
            acc2[r] = 0.0f;
            acc1[r] = 0.0f;
            acc0[r] = 0.0f;
        }
    };

    // Packed weight limbs of the 16 (pixel, bin) results of one axis; cb is
    // the bin's constant (bin_const).
    auto weights = [&](const f32x16 &ah, const f32x16 &al, uint32_t cb, uint32_t (&e)[16]) {
#pragma unroll
        for (int r = 0; r < 16; r++) e[r] = s_wt[(s1_bits(ah[r], al[r], cb) >> 15) & (kWKeys - 1)];
    };

    // One tile of up to 32 pixels (queue slot m = lane & 31) from prefetched
    // input; `next` reuses the input registers once they are converted.
    auto tile = [&](RawSlices<T, F> &raw, int nvalid, auto next) {
        float n2x = 0.0f, n2y = 0.0f;
        f16x8 X[KS], Y[KS];
        raw.convert(0, X, n2x);
        raw.convert(1, Y, n2y);
        next();
        n2x += __shfl_xor(n2x, 32);
        n2y += __shfl_xor(n2y, 32);
        if (g == 0) {
            const PixelInit ix = pixel_init(n2x), iy = pixel_init(n2y);
            ini[ln] = ix.a;
            ini[32 + ln] = ix.l;
            ini[64 + ln] = iy.a;
            ini[96 + ln] = iy.l;
        }
        uint32_t ex[16], ey[16];
        {
            f16x8 ph[KS], pl[KS];
#pragma unroll
            for (int j = 0; j < KS; j++) {
                ph[j] = palette_operand(s_pop, 0, 0, j, lane);
                pl[j] = palette_operand(s_pop, 0, 1, j, lane);
            }
            f32x16 ah = row_init(ini, g), al = row_init(ini + 32, g);
            axis_dot<KS, true>(X, ph, pl, ah, al);
            weights(ah, al, cbx, ex);
        }
        {
            f16x8 ph[KS], pl[KS];
#pragma unroll
            for (int j = 0; j < KS; j++) {
                ph[j] = palette_operand(s_pop, 1, 0, j, lane);
                pl[j] = palette_operand(s_pop, 1, 1, j, lane);
            }
            f32x16 ah = row_init(ini + 64, g), al = row_init(ini + 96, g);
            axis_dot<KS, true>(Y, ph, pl, ah, al);
            weights(ah, al, cby, ey);
        }
        if (nvalid < 32) {        // pixels past the end of the list vote nothing
            // (kept a real branch: only the last tile of a round is partial)
            __asm__ volatile("" ::: "memory");
#pragma unroll
            for (int r = 0; r < 16; r++)
                if (acc_row(r, g) >= nvalid) ex[r] = 0u;
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

    int t = t0 + wv;
    ListCursor cur_list;
    cur_list.start(list, s_pref, nslices, slice_px, t < tend ? 32 * t : 0);
    // lane m of tile tt: entry 32 tt + m, or the tile's first entry past the end
    auto pixel = [&](int tt) { return cur_list.pixel(32 * tt + ln < n ? 32 * tt + ln : 32 * tt); };
    // the next tile's rows are loaded as soon as the current ones are converted
    RawSlices<T, F> raw;
    int tn = tend, idx = 0;                            // next tile, and this lane's pixel in it
    if (t < tend) {
        raw.load(emb + (size_t)pixel(t) * dstride, yoff, g);
        tn = take_tile(s_next, lane, t0, kWpb);
        if (tn < tend) idx = pixel(tn);
    }
    while (t < tend) {
        int tnn = tend;
        tile(raw, min(32, n - 32 * t), [&]() {
            if (tn < tend) {
                raw.load(emb + (size_t)idx * dstride, yoff, g);
                tnn = take_tile(s_next, lane, t0, kWpb);
                if (tnn < tend) idx = pixel(tnn);
            }
        });
        t = tn;
        tn = tnn;
    }
    fold();

    // one global atomic per bin of the grid
    __syncthreads();
    const int nb = Bw * Bh;
    unsigned long long *dst = hrep + (size_t)(blockIdx.x % kReplicas) * nb;
    for (int i = tid; i < kMfmaBins * kMfmaBins; i += blockDim.x) {
        const int b = i / kMfmaBins, a = i % kMfmaBins;
        const unsigned long long v = s_h[b * kHStride + a];
        if (a < Bw && b < Bh && v) atomicAdd(dst + b * Bw + a, v);
    }
    if (blockIdx.x == 0)
        for (int k = tid; k < cap; k += blockDim.x) cents[k].npix = 0;
}

// ---------------------------------------------------------------------------
// Pass 2: assignment + label write-out
// ---------------------------------------------------------------------------
// LDS bytes of k_assign_mfma: code table, palette operands, bin constants,
// candidate batches, bin -> centroid table, counts, per wave x keys and y
// keys [32 bins][kKeyStride] (u32), then the peak-extraction state.
constexpr size_t kAssignLdsCore = (size_t)kCKeys * 2 + kPopBytes + 4 * kMfmaBins * 4 + (size_t)kMaxBatchLds * 20 +
                                  kMfmaBins * kMfmaBins * 2 + kMfmaBins * kMfmaBins * 4 +
                                  (size_t)kWpb2 * 2 * kMfmaBins * kKeyStride * 4 + sizeof(PeakLds) +
                                  (kMaxSlices + 1) * 4 + 16;
// then, 16-byte aligned, per wave the 32 search results of a tile, and the
// summed vote histogram (32 x 32 slots)
constexpr size_t kBestOff = (kAssignLdsCore + 15) & ~(size_t)15;
constexpr size_t kSumOff = kBestOff + (size_t)kWpb2 * 32 * 4;
constexpr size_t kAssignLds = kSumOff + (size_t)kMfmaBins * kMfmaBins * 8;

// Every workgroup first sums the vote histograms `hcur` of the vote launch
// and extracts the peaks in LDS (identical in every workgroup); workgroup 0
// writes the centroid records (all fields but the pixel count), K and the
// summed histogram `hlast`, and the grid clears `hzero`, the histograms the
// next frame's vote launch accumulates into.
//
// Then, per tile of 32 pixels, the distance codes of both axes for the
// candidate slots (palette entries of the slots' bins as the MFMA rows, so
// that each lane holds one pixel and 16 slots) go to LDS as search keys:
// x key (c_x << 16) | column slot and y key (c_y << 16) | 128 row slot, laid
// out [slot][kKeyStride] so that lane m reads pixel m's key of any slot at a
// fixed stride.  The low halves are written once; per tile only the codes
// are stored, as 16-bit writes.  The candidate search walks the batches of 4
// columns of one row (see the search below).  The sum of an x key and a y
// key is ((c_x + c_y) << 16) | (128 row slot + column slot), taken with
// unsigned saturation: codes are below 2^16 but a sum of two may not be.
// The minimum is exact unless every candidate saturates (all code sums of
// the pixel at least 2^16); such a pixel is searched again in 64 bits.
template <typename T, int F>
__global__ __launch_bounds__(kWpb2 * 64) __attribute__((amdgpu_waves_per_eu(kWpb2 / 4))) void k_assign_mfma(
    const T *__restrict__ emb, int32_t dstride, int32_t yoff, const int32_t *__restrict__ list,
    const int32_t *__restrict__ counts, int32_t nslices, int32_t slice_px, int32_t npix, uint32_t tau_code, Tables tb,
    const unsigned long long *__restrict__ hcur, unsigned long long *__restrict__ hzero,
    unsigned long long *__restrict__ hlast, int32_t Bw, int32_t Bh, long long cut, int32_t cap,
    cpe_centroid *__restrict__ cents, int32_t *__restrict__ num, int32_t *__restrict__ labels,
    float *__restrict__ score_map)
{
    constexpr int KS = AxisShape<F>::KS;
    constexpr int kThreads = kWpb2 * 64;
    static_assert(kThreads >= kPeakThreads, "the peak prologue takes two histogram slots per thread");
    static_assert(kAssignLds <= 160 * 1024, "LDS of one compute unit");
    // All LDS is static, so that table addresses are compile-time constants.
    __shared__ __align__(16) unsigned char smem[kAssignLds];
    uint16_t *s_ct = reinterpret_cast<uint16_t *>(smem);                            // [kCKeys]
    uint32_t *s_pop = reinterpret_cast<uint32_t *>(s_ct + kCKeys);                  // palette operands
    uint32_t *s_cb = s_pop + kPopBytes / 4;                                          // [2][32] bin_const by bin
    uint32_t *s_cbs = s_cb + 2 * kMfmaBins;                                           // [2][32] by slot
    u32x4 *s_bo = reinterpret_cast<u32x4 *>(s_cbs + 2 * kMfmaBins);                // [kMaxBatchLds]
    uint32_t *s_bh = reinterpret_cast<uint32_t *>(s_bo + kMaxBatchLds);             // [kMaxBatchLds]
    uint16_t *s_rank = reinterpret_cast<uint16_t *>(s_bh + kMaxBatchLds);           // [32 * 32]
    int32_t *s_cnt = reinterpret_cast<int32_t *>(s_rank + kMfmaBins * kMfmaBins);   // [1024]
    uint32_t *s_keys = reinterpret_cast<uint32_t *>(s_cnt + kMfmaBins * kMfmaBins); // [kWpb2][2][32][kKeyStride]
    PeakLds &pl = *reinterpret_cast<PeakLds *>(s_keys + kWpb2 * 2 * kMfmaBins * kKeyStride);
    int *s_pref = reinterpret_cast<int *>(&pl + 1);                                  // [kMaxSlices + 1]
    int *s_next = s_pref + kMaxSlices + 1;                                            // next tile of the run
    uint32_t *s_best = reinterpret_cast<uint32_t *>(smem + kBestOff);                 // [kWpb2][32]
    unsigned long long *s_h = reinterpret_cast<unsigned long long *>(smem + kSumOff);  // [32 * 32] summed votes

    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int g = lane >> 5, ln = lane & 31;
    const int nb = Bw * Bh;

    PeakLoad pld;                                   // issued before the table staging
    peaks_lds_load(hcur, Bw, Bh, pld);
    // This wave's search keys, [bin][kKeyStride] per axis: x key of bin a,
    // pixel m at kx[a * kKeyStride + m], y key of bin b at ky[...]; their
    // low halves (a for x keys, 128 b for y keys) are written here, while
    // the loads are in flight, and the codes fill the high halves per tile.
    uint32_t *kx = s_keys + wv * 2 * kMfmaBins * kKeyStride;
    uint32_t *ky = kx + kMfmaBins * kKeyStride;
    {
        constexpr int kVecPerRow = kKeyStride / 4;
#pragma unroll
        for (int i = lane; i < 2 * kMfmaBins * kVecPerRow; i += 64) {
            const int row = i / kVecPerRow;          // a power-of-two division: a shift
            const uint32_t v = row < kMfmaBins ? (uint32_t)row : 128u * (uint32_t)(row - kMfmaBins);
            const u32x4 v4 = {v, v, v, v};
            reinterpret_cast<u32x4 *>(kx)[i] = v4;
        }
    }
    SliceLoad sl;
    if (list) slice_load(counts, nslices, sl);
    {
        constexpr int kN = kCKeys / 8, kPer = (kN + kThreads - 1) / kThreads;
        u32x4 w[kPer];
#pragma unroll
        for (int k = 0; k < kPer; k++) {
            const int i = k * kThreads + tid;
            w[k] = reinterpret_cast<const u32x4 *>(tb.ct_pm)[i < kN ? i : 0];
        }
#pragma unroll
        for (int k = 0; k < kPer; k++) {
            const int i = k * kThreads + tid;
            if (i < kN) reinterpret_cast<u32x4 *>(s_ct)[i] = w[k];
        }
        for (int i = tid; i < kPopBytes / 16; i += kThreads)
            reinterpret_cast<u32x4 *>(s_pop)[i] = reinterpret_cast<const u32x4 *>(tb.pop)[i];
        if (tid < 2 * kMfmaBins)
            s_cb[tid] = bin_const(tid < kMfmaBins ? tb.np1_x[tid] : tb.np1_y[tid - kMfmaBins]);
    }
    for (int i = tid; i < kMfmaBins * kMfmaBins; i += kThreads) s_cnt[i] = 0;
    if (tid == 0) *s_next = 0;
    peaks_lds_sum(pld, s_h, pl);
    if (list) slice_scan(sl, nslices, s_pref);
    __syncthreads();

    // the workgroup's run of tiles of 32 list entries; the first tile's list
    // entries and rows are loaded while the peaks are extracted
    const int n = list ? s_pref[nslices] : npix, ntiles = (n + 31) >> 5;
    int t0, tend;
    block_run(ntiles, blockIdx.x, gridDim.x, t0, tend);
    int t = t0 + wv;
    ListCursor cur_list;
    cur_list.start(list, s_pref, nslices, slice_px, t < tend ? 32 * t : 0);
    // lane m of tile tt: entry 32 tt + m, or the tile's first entry past the end
    auto pixel = [&](int tt) { return cur_list.pixel(32 * tt + ln < n ? 32 * tt + ln : 32 * tt); };
    RawSlices<T, F> raw;
    int ip = t < tend ? pixel(t) : 0;                   // this lane's pixel in this tile
    peaks_lds_find(Bw, Bh, cut, cap, s_h, pl, s_bo, s_bh, s_rank, s_cb, s_cbs, [&]() {
        if (t < tend) raw.load(emb + (size_t)ip * dstride, yoff, g);
    });
    const int Kc = pl.Kc;
    if (blockIdx.x == 0) {
        for (int k = tid; k < Kc; k += kThreads) {
            const int i = pl.pk[k], a = i & 31, b = i >> 5;
            cpe_centroid *c = cents + k;    // npix was reset by the vote launch and is counted below
            c->bin_x = a;
            c->bin_y = b;
            c->x = tb.cx[a];
            c->y = tb.cy[b];
            c->score = (double)s_h[i] * 0x1p-30;
            c->reserved = 0;
        }
        for (int i = tid; i < nb; i += kThreads) hlast[i] = s_h[(i / Bw) * 32 + i % Bw];
        if (tid == 0) *num = pl.K;
    }
    for (int i = blockIdx.x * kThreads + tid; i < kReplicas * nb; i += gridDim.x * kThreads) hzero[i] = 0ull;

    if (Kc == 0) {              // no centroid: every participating pixel is unlabelled
        ListCursor c0;
        c0.start(list, s_pref, nslices, slice_px, 32 * t0 + 64 * wv < n ? 32 * t0 + 64 * wv : 0);
        for (int i = 32 * t0 + tid; i < min(32 * tend, n); i += kThreads) {
            const int p = c0.pixel(i);
            labels[p] = 0;
            if (score_map) score_map[p] = 0.0f;
        }
        return;
    }
    const int nbat = min(pl.nbat, kMaxBatchLds);    // a multiple of kBatchPad


    // The MFMA rows are the candidate slots: the palette operands of slot j's
    // bin, gathered once and kept in registers for the whole run; codes are
    // computed only for the groups of 8 slots that hold candidates.
    const int nslot[2] = {__builtin_amdgcn_readfirstlane(pl.ncol), __builtin_amdgcn_readfirstlane(pl.nrow)};
    f16x8 pop_h[2][KS], pop_l[2][KS];
#pragma unroll
    for (int ax = 0; ax < 2; ax++) {
        const int bin = ax ? pl.rowbin[ln] : pl.colbin[ln];
#pragma unroll
        for (int j = 0; j < KS; j++) {
            pop_h[ax][j] = palette_operand(s_pop, ax, 0, j, g * 32 + bin);
            pop_l[ax][j] = palette_operand(s_pop, ax, 1, j, g * 32 + bin);
        }
    }

    // Codes of one tile into the keys' high halves (pixel m = lane & 31; this
    // lane's 16 bins acc_row(r, g) of each axis); `next` reuses the input
    // registers once they are converted.
    auto codes = [&](RawSlices<T, F> &raw, auto next) {
        float n2x = 0.0f, n2y = 0.0f;
        f16x8 X[KS], Y[KS];
        raw.convert(0, X, n2x);
        raw.convert(1, Y, n2y);
        next();
        // the pixel's part of the constant: 256 |Xr|^2, the accumulators
        // starting at kMagic (one starting value shared by all four)
        const uint32_t npx = (uint32_t)(n2x + __shfl_xor(n2x, 32)) << 8;
        const uint32_t npy = (uint32_t)(n2y + __shfl_xor(n2y, 32)) << 8;
#pragma unroll
        for (int ax = 0; ax < 2; ax++) {
            f32x16 ah, al;
#pragma unroll
            for (int r = 0; r < 16; r++) {
                ah[r] = kMagic;
                al[r] = kMagic;
            }
            axis_dot<KS, false>(ax ? Y : X, pop_h[ax], pop_l[ax], ah, al);
            const uint32_t np = ax ? npy : npx;
            // high half of key (slot acc_row(r, g), pixel ln)
            uint16_t *dst = reinterpret_cast<uint16_t *>((ax ? ky : kx) + 4 * g * kKeyStride + ln) + 1;
#pragma unroll
            for (int r4 = 0; r4 < 4; r4++) {
                if (8 * r4 >= nslot[ax]) break;      // wave-uniform: no candidate in slots 8 r4 ..
                const u32x4 cb = *reinterpret_cast<const u32x4 *>(s_cbs + ax * kMfmaBins + 8 * r4 + 4 * g);
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const int r = 4 * r4 + i;
                    dst[2 * kKeyStride * (8 * r4 + i)] = s_ct[(s1_bits(ah[r], al[r], np + cb[i]) >> 14) & (kCKeys - 1)];
                }
            }
        }
    };

    // Candidate search.  Lane l serves the four pixels 4 q .. 4 q + 3
    // (q = l & 7) for the batches j, j + 8, ... (j = l >> 3): one 16-byte
    // read fetches a column's keys of its four pixels, so each address
    // computation and each read serve four pixels.  The eight lanes of a
    // pixel quad then combine their minima, and lane m takes pixel m's
    // result through LDS; lanes of half 0 write the labels of valid pixels.
    uint32_t *best_w = s_best + wv * 32;
    auto search = [&](int pix, int nvalid) {
        __builtin_amdgcn_wave_barrier();
        const int q = lane & 7, j0 = lane >> 3;
        const unsigned char *kxq = reinterpret_cast<const unsigned char *>(kx + 4 * q);
        const unsigned char *kyq = reinterpret_cast<const unsigned char *>(ky + 4 * q);
        uint32_t b4[4] = {0xffffffffu, 0xffffffffu, 0xffffffffu, 0xffffffffu};
#pragma unroll 2
        for (int bi = j0; bi < nbat; bi += 8) {     // nbat is a multiple of 8: the same count for every lane
            const u32x4 o = s_bo[bi];
            const uint32_t hb = s_bh[bi];
            const u32x4 v0 = *reinterpret_cast<const u32x4 *>(kxq + o.x);
            const u32x4 v1 = *reinterpret_cast<const u32x4 *>(kxq + o.y);
            const u32x4 v2 = *reinterpret_cast<const u32x4 *>(kxq + o.z);
            const u32x4 v3 = *reinterpret_cast<const u32x4 *>(kxq + o.w);
            const u32x4 yk = *reinterpret_cast<const u32x4 *>(kyq + hb);
#pragma unroll
            for (int e = 0; e < 4; e++)
                b4[e] = min(b4[e], __builtin_elementwise_add_sat((uint32_t)min(min(v0[e], v1[e]), min(v2[e], v3[e])),
                                                                 yk[e]));
        }
#pragma unroll
        for (int e = 0; e < 4; e++) {
            b4[e] = min(b4[e], (uint32_t)__shfl_xor((int)b4[e], 8));
            b4[e] = min(b4[e], (uint32_t)__shfl_xor((int)b4[e], 16));
            b4[e] = min(b4[e], (uint32_t)__shfl_xor((int)b4[e], 32));
        }
        if (lane < 8) {
            const u32x4 w4 = {b4[0], b4[1], b4[2], b4[3]};
            *reinterpret_cast<u32x4 *>(best_w + 4 * q) = w4;
        }
        __builtin_amdgcn_wave_barrier();
        const uint32_t best = best_w[ln];
        const unsigned char *kxl = reinterpret_cast<const unsigned char *>(kx + ln);
        const unsigned char *kyl = reinterpret_cast<const unsigned char *>(ky + ln);
        uint32_t sum = best >> 16, idx = best & 0xffffu;   // code sum and 128 (row slot) + column slot
        if (best == 0xffffffffu) {   // every sum saturated: all batches again, in 64 bits
            unsigned long long b64 = ~0ull;
            for (int bi = 0; bi < nbat; bi++) {
                const u32x4 o = s_bo[bi];
                const unsigned long long yk = *reinterpret_cast<const uint32_t *>(kyl + s_bh[bi]);
#pragma unroll
                for (int c = 0; c < 4; c++)
                    b64 = min(b64, (unsigned long long)*reinterpret_cast<const uint32_t *>(kxl + o[c]) + yk);
            }
            sum = (uint32_t)(b64 >> 16);
            idx = (uint32_t)b64 & 0xffffu;
        }
        if (g == 0 && ln < nvalid) {
            if (sum < tau_code) {      // Eq8 (tau_code = ceil(4096 tau))
                const int a = pl.colbin[idx & 31u], b = pl.rowbin[(idx >> 7) & 31u];
                const int k = s_rank[b * kMfmaBins + a] & (kMfmaBins * kMfmaBins - 1);
                labels[pix] = k + 1;
                if (score_map) score_map[pix] = expf(-((float)sum * 0x1p-12f));
                atomicAdd(s_cnt + k, 1);
            } else {
                labels[pix] = 0;
                if (score_map) score_map[pix] = 0.0f;
            }
        }
        __builtin_amdgcn_wave_barrier();
    };

    // the next tile's rows are loaded as soon as the current ones are converted
    int tn = tend, ipn = 0;                             // next tile; this lane's pixel in it
    if (t < tend) {
        tn = take_tile(s_next, lane, t0, kWpb2);
        if (tn < tend) ipn = pixel(tn);
    }
    while (t < tend) {
        int tnn = tend, ipnn = 0;
        codes(raw, [&]() {
            if (tn < tend) {
                raw.load(emb + (size_t)ipn * dstride, yoff, g);
                tnn = take_tile(s_next, lane, t0, kWpb2);
                if (tnn < tend) ipnn = pixel(tnn);
            }
        });
        search(ip, min(32, n - 32 * t));
        t = tn;
        tn = tnn;
        ip = ipn;
        ipn = ipnn;
    }
    __syncthreads();
    for (int i = tid; i < Kc && i < kMfmaBins * kMfmaBins; i += kThreads)
        if (s_cnt[i]) atomicAdd(&cents[i].npix, s_cnt[i]);
}

}  // namespace cpe
