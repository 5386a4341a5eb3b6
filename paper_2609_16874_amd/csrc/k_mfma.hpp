// k_mfma.hpp -- matrix-core decoder kernels: the vote for every bin grid (in
// passes over blocks of 32 x 32 bins), the assignment for grids up to 32 x 32.
//
// Both passes stream a compact list of participating pixels (or every
// pixel, when the frame has no foreground channel), cut into tiles of 32
// consecutive entries.  The assignment, and the vote of three-launch
// frames, read the list in global memory (written by k_compact, or by the
// vote launch in two-launch frames): every workgroup gets a contiguous run
// of tiles of the same length to within one.  In two-launch frames the vote
// lists its own share of the pixels in LDS (FusedArgs).  The waves take
// their tiles one at a time from a counter in LDS (so that they finish
// together however the SIMDs favour older waves), always loading the
// embedding rows of the next tile (and the list entries of the one after)
// before computing the current one.  Every tile but the last is full.
//
// Per-axis distances (Eq4/Eq10).  The input X = rint(4096 v) (|X| <= 6144)
// is split into int8 limbs X = 128 Xh + Xl (|Xh| <= 48, |Xl| <= 64) and the
// palette into -2P = 128 hi + lo (|hi| <= 64, |lo| <= 64), so that
//   S = |X|^2 + |P|^2 + 2^14 Xh.hi + 2^7 (Xh.lo + Xl.hi) + Xl.lo
// with three dense [pixels x channels] x [channels x bins] contractions on
// v_mfma_i32_32x32x32_i8 (exact int32 accumulation; the middle one takes two
// instructions, or all three share one pixel operand when 2F <= 16, see
// AxisOp); S < 2^32 follows modulo 2^32 from two shift-and-add instructions.
// |X|^2 is three int8 dot products of the limbs.
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
// holds one pixel and 16 slots, and distances are computed for the groups of
// 8 slots that hold candidates: r = sqrtf(fl32(S)) correctly rounded, stored
// in LDS as binary32 bits (which order like the distances, r >= 0).  The
// candidate search walks batches of 4 columns of one row, in (row, column)
// order: the smallest x distance of the batch plus the row's y distance is
// summed exactly in binary64, the batch index fills the low bits of that sum
// (always zero there), and one binary64 minimum selects the smallest distance
// sum and, on ties, the first batch; within it the first column attaining
// the batch's x minimum wins.  Slots keep the bins' order, so this is the
// lowest centroid index among the smallest sums.
#pragma once

#include <type_traits>

#include "cpe_common.hpp"
#include "k_compact.hpp"
#include "k_peaks.hpp"

namespace cpe {

typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x16 __attribute__((ext_vector_type(16)));

constexpr int kPopBytes = 2 * kPopKinds * 64 * 16;   // palette operands of both axes

// The int8 operand of one axis of one pixel, for the lane of half g = lane >> 5
// of the MFMA, which holds the 16 K slots 16 g .. 16 g + 15.  The lane's
// channels are c_b = 8 g + b and, for 2F > 16, 16 + 8 g + b (b = 0..7;
// channels past 2F are zero).
//   2F > 16: a[0] = Xh of the 16 channels, a[1] = Xl; with the palette
//            operand kinds 0 = hi and 1 = lo (same channel order):
//            Xh.hi, Xh.lo + Xl.hi, Xl.lo in four MFMAs;
//   2F <= 16: a[0] = Xh of the 8 channels, then their Xl; with the kinds
//            0 = (hi, 0), 1 = (lo, hi), 2 = (0, lo) the three products take
//            one MFMA each.
template <int F>
struct AxisOp {
    static constexpr bool kPacked = 2 * F <= 16;
    static constexpr int N = kPacked ? 1 : 2;
    i32x4 a[N];
};

__device__ __forceinline__ i32x16 mfma8(i32x4 a, i32x4 b, i32x16 c)
{
    return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 mfma16(f16x8 a, f16x8 b, f32x16 c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// Steps (binary32 units in the last place) by which the fast assignment
// search needs the second smallest batch sum to exceed the smallest: at
// least 7 by its error bound (see k_assign_mfma).
constexpr int kFastGap = 8;

// Row of the 32 x 32 MFMA result held by register r of a lane in group g.
__device__ __forceinline__ constexpr int acc_row(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }

// int8 limbs of two channels: Xh = rint(32 c) and Xl = rint(128 (32 c - Xh)),
// c = clamp(v, -1.5, 1.5), so that 128 Xh + Xl = rint(4096 c) (128 Xh is
// even, so the ties agree).  In fp16: 32 c + 1536 lies in [1488, 1584], where
// the spacing is 1, so the fused multiply-add rounds it to 1536 + Xh; 32 c -
// Xh is exact (|.| <= 1/2) and 128 times it plus 1536 rounds to 1536 + Xl.
// The low byte of each result's bit pattern 0x6600 + k is k as an int8.  A
// NaN clamps to -1.5 (max returns the non-NaN operand).
struct LimbPair {
    uint32_t h, l;     // two fp16 bit patterns each
};
__device__ __forceinline__ LimbPair limbs_f16(f16x2 v)
{
    const f16x2 lo = {(_Float16)-1.5f, (_Float16)-1.5f}, hi = {(_Float16)1.5f, (_Float16)1.5f};
    const f16x2 k32 = {(_Float16)32.0f, (_Float16)32.0f}, k128 = {(_Float16)128.0f, (_Float16)128.0f};
    const f16x2 m = {(_Float16)1536.0f, (_Float16)1536.0f};
    f16x2 c = __builtin_elementwise_max(v, lo);
    c = __builtin_elementwise_min(c, hi);
    const f16x2 h = __builtin_elementwise_fma(c, k32, m);
    const f16x2 hv = h - m;
    const f16x2 d = __builtin_elementwise_fma(c, k32, -hv);
    const f16x2 l = __builtin_elementwise_fma(d, k128, m);
    return {__builtin_bit_cast(uint32_t, h), __builtin_bit_cast(uint32_t, l)};
}

// The same in fp32 (exact: |32 c| < 2^22 around 1.5 * 2^23, whose spacing is
// 1); the low byte of the bit pattern 0x4B400000 + k is k as an int8.
__device__ __forceinline__ void limbs_f32(float v, uint32_t &h, uint32_t &l)
{
    constexpr float kM = 12582912.0f;
    const float c = fminf(fmaxf(v, -1.5f), 1.5f);
    const float hf = __builtin_fmaf(c, 32.0f, kM);
    const float hv = hf - kM;
    const float d = __builtin_fmaf(c, 32.0f, -hv);
    const float lf = __builtin_fmaf(d, 128.0f, kM);
    h = __float_as_uint(hf);
    l = __float_as_uint(lf);
}

// Low bytes of the two halves of w0 (bytes 0, 1 of the result) and of w1
// (bytes 2, 3).
__device__ __forceinline__ uint32_t low_bytes(uint32_t w1, uint32_t w0)
{
    return __builtin_amdgcn_perm(w1, w0, 0x06040200u);
}

// Raw input words of one lane's operand slices: for each axis and K-step j
// the 8 channels [16 j + 8 g, 16 j + 8 g + 8) of one pixel's axis block
// (channels past 2F read as 0).  Loaded one tile ahead of their use.
template <typename T, int F>
struct RawSlices {
    static constexpr int C = 2 * F;
    static constexpr int KS = (C + 15) / 16;
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

    // int8 operand of one axis and this lane's part of |X|^2 over its
    // channels (added to n2).
    __device__ __forceinline__ void convert(int ax, AxisOp<F> &op, int &n2) const
    {
        uint32_t hb[KS][2], lb[KS][2];      // packed limb bytes, 4 channels per word
#pragma unroll
        for (int j = 0; j < KS; j++) {
            if constexpr (kH && kVec) {
                LimbPair p[4];
#pragma unroll
                for (int q = 0; q < 4; q++) p[q] = limbs_f16(__builtin_bit_cast(f16x2, w[ax][j][q]));
#pragma unroll
                for (int q = 0; q < 2; q++) {
                    hb[j][q] = low_bytes(p[2 * q + 1].h, p[2 * q].h);
                    lb[j][q] = low_bytes(p[2 * q + 1].l, p[2 * q].l);
                }
            } else {
                uint32_t h[8], l[8];
#pragma unroll
                for (int s = 0; s < 8; s++) limbs_f32(__uint_as_float(w[ax][j][s]), h[s], l[s]);
#pragma unroll
                for (int q = 0; q < 2; q++) {
                    hb[j][q] = low_bytes(__builtin_amdgcn_perm(h[4 * q + 3], h[4 * q + 2], 0x05040100u),
                                         __builtin_amdgcn_perm(h[4 * q + 1], h[4 * q], 0x05040100u));
                    lb[j][q] = low_bytes(__builtin_amdgcn_perm(l[4 * q + 3], l[4 * q + 2], 0x05040100u),
                                         __builtin_amdgcn_perm(l[4 * q + 1], l[4 * q], 0x05040100u));
                }
            }
        }
        int hh = 0, hl = 0, ll = 0;
#pragma unroll
        for (int j = 0; j < KS; j++)
#pragma unroll
            for (int q = 0; q < 2; q++) {
                hh = __builtin_amdgcn_sdot4((int)hb[j][q], (int)hb[j][q], hh, false);
                hl = __builtin_amdgcn_sdot4((int)hb[j][q], (int)lb[j][q], hl, false);
                ll = __builtin_amdgcn_sdot4((int)lb[j][q], (int)lb[j][q], ll, false);
            }
        n2 += (hh << 14) + (hl << 8) + ll;
        if constexpr (AxisOp<F>::kPacked) {
            op.a[0] = i32x4{(int)hb[0][0], (int)hb[0][1], (int)lb[0][0], (int)lb[0][1]};
        } else {
            op.a[0] = i32x4{(int)hb[0][0], (int)hb[0][1], (int)hb[1][0], (int)hb[1][1]};
            op.a[1] = i32x4{(int)lb[0][0], (int)lb[0][1], (int)lb[1][0], (int)lb[1][1]};
        }
    }
};


// An empty asm that takes the converted operands and clobbers memory: the
// next tile's row loads, which follow it, issue after the conversion and
// reuse the input registers (otherwise the compiler hoists them above the
// conversion and copies 16 registers per tile).
template <int F>
__device__ __forceinline__ void after_convert(AxisOp<F> &X, AxisOp<F> &Y, int &n2x, int &n2y)
{
    if constexpr (AxisOp<F>::kPacked)
        __asm__ volatile("" : "+v"(X.a[0]), "+v"(Y.a[0]), "+v"(n2x), "+v"(n2y) : : "memory");
    else
        __asm__ volatile("" : "+v"(X.a[0]), "+v"(X.a[1]), "+v"(Y.a[0]), "+v"(Y.a[1]), "+v"(n2x), "+v"(n2y) : : "memory");
}

// Palette operand of kind k for axis ax of lane `lane` (bin lane & 31, K
// slots 16 (lane >> 5) .. + 15).
__device__ __forceinline__ i32x4 palette_operand(const uint32_t *__restrict__ pop, int ax, int k, int lane)
{
    return *reinterpret_cast<const i32x4 *>(pop + (((ax * kPopKinds + k) * 64 + lane) * 4));
}

// Word group i (16 bytes) of the LDS palette operands [axis][kind][64][16] for
// the x bins of block bx and the y bins of block by, from the table
// [axis][kMaxBinBlocks][kind][64][16].
__device__ __forceinline__ u32x4 pop_block(const uint32_t *__restrict__ pop, int i, int bx, int by)
{
    constexpr int kAxis = kPopKinds * 64;                 // 16-byte groups per axis and block
    const int ax = i / kAxis, r = i % kAxis;
    const int blk = ax ? by : bx;
    return reinterpret_cast<const u32x4 *>(pop)[(ax * kMaxBinBlocks + blk) * kAxis + r];
}

// The three limb products of one axis: hh = Xh.hi, mid = Xh.lo + Xl.hi and
// ll = ll0 + Xl.lo (ll0: the starting values).  PIX_ROWS: pixels are the
// MFMA rows (pass 1) or its columns (pass 2).
template <int F, bool PIX_ROWS>
__device__ __forceinline__ void axis_products(const AxisOp<F> &X, const i32x4 (&P)[kPopKinds], i32x16 ll0,
                                              i32x16 &hh, i32x16 &mid, i32x16 &ll)
{
    const i32x16 z = {};
    auto mm = [](i32x4 px, i32x4 pal, i32x16 c) { return PIX_ROWS ? mfma8(px, pal, c) : mfma8(pal, px, c); };
    if constexpr (AxisOp<F>::kPacked) {
        hh = mm(X.a[0], P[0], z);
        mid = mm(X.a[0], P[1], z);
        ll = mm(X.a[0], P[2], ll0);
    } else {
        hh = mm(X.a[0], P[0], z);
        mid = mm(X.a[0], P[1], z);
        mid = mm(X.a[1], P[0], mid);
        ll = mm(X.a[1], P[1], ll0);
    }
}

// 2^14 hh + 2^7 mid + ll + c (mod 2^32) as two shift-and-add instructions
// and one add.
__device__ __forceinline__ uint32_t assemble(int hh, int mid, int ll, uint32_t c)
{
    const uint32_t t = ((uint32_t)hh << 7) + (uint32_t)mid;
    return (t << 7) + (uint32_t)ll + c;
}

// Starting values of one accumulator for the 16 rows acc_row(r, g) of a lane
// in group g, from an LDS array indexed by row.
__device__ __forceinline__ i32x16 row_init(const uint32_t *a, int g)
{
    i32x16 v;
#pragma unroll
    for (int r4 = 0; r4 < 4; r4++) {
        const u32x4 w = *reinterpret_cast<const u32x4 *>(a + 8 * r4 + 4 * g);
#pragma unroll
        for (int i = 0; i < 4; i++) v[4 * r4 + i] = (int)w[i];
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
// Pass 1: recovery + soft voting
// ---------------------------------------------------------------------------
// Row stride (in 64-bit words) of the vote kernel's LDS histogram: one word
// of padding per row puts the 32 rows that one fold instruction touches
// (lanes = y bins, fixed x bin) into distinct banks.
constexpr int kHStride = kMfmaBins + 1;

// LDS bytes of k_vote_mfma: the packed weight table, the 64-bit histogram,
// the palette operands, per wave |X|^2 of one tile's pixels per axis, the
// slice prefix sums and counters; with the compaction folded in (FUSED),
// the workgroup's own participating pixels.
constexpr size_t kVoteLds(int wpb, bool fused)
{
    return (size_t)kWKeys * 4 + kMfmaBins * kHStride * 8 + kPopBytes + (size_t)wpb * 64 * 4 + (kMaxSlices + 1) * 4 +
           16 + (fused ? (size_t)kFusedMaxSeg * 4 : 0);
}

// Eight foreground values from pixel p0 on (p0 a multiple of 8), in two
// parts: load8_raw issues one (fp16) or two (fp32) 16-byte loads when the
// plane is 16-byte aligned and the eight lie below lim (zero words
// otherwise); load8_values gives the values, loading pixel by pixel below
// lim (0 beyond) where the vector loads do not apply.
template <typename T>
struct Raw8 {
    uint4 w[sizeof(T) / 2];
};
template <typename T>
__device__ __forceinline__ Raw8<T> load8_raw(const T *fg, int p0, int lim, bool vec)
{
    Raw8<T> r = {};
    if (vec && p0 + 8 <= lim) {
#pragma unroll
        for (int k = 0; k < (int)(sizeof(T) / 2); k++) r.w[k] = reinterpret_cast<const uint4 *>(fg + p0)[k];
    }
    return r;
}
template <typename T>
__device__ __forceinline__ void load8_values(const T *fg, int p0, int lim, bool vec, const Raw8<T> &r, float v[8])
{
    if (vec && p0 + 8 <= lim) {
        if constexpr (sizeof(T) == 2) {
            const uint32_t ww[4] = {r.w[0].x, r.w[0].y, r.w[0].z, r.w[0].w};
#pragma unroll
            for (int i = 0; i < 4; i++) {
                v[2 * i] = half_bits_to_float(ww[i] & 0xffffu);
                v[2 * i + 1] = half_bits_to_float(ww[i] >> 16);
            }
        } else {
#pragma unroll
            for (int k = 0; k < 2; k++) {
                v[4 * k] = __uint_as_float(r.w[k].x);
                v[4 * k + 1] = __uint_as_float(r.w[k].y);
                v[4 * k + 2] = __uint_as_float(r.w[k].z);
                v[4 * k + 3] = __uint_as_float(r.w[k].w);
            }
        }
    } else {
#pragma unroll
        for (int i = 0; i < 8; i++) v[i] = fg && p0 + i < lim ? load_scalar<T>(fg + p0 + i) : 0.0f;
    }
}

// The compaction folded into the vote launch (frames of up to kFusedMaxPixels
// pixels, grids up to 32 x 32).  Workgroup b lists the participating pixels
// twice: those of its range b * seg_cap .. (b + 1) * seg_cap - 1 of the
// frame (seg_cap a multiple of 8) into list[b * seg_cap ..], their number
// into counts[b] -- the assignment launch reads these segments as its slices,
// in the frame's order -- and those of the slices of `slice` pixels (a
// multiple of 64) dealt to it in turn, in LDS, in any order: the pixels it
// votes on, spread over the frame so that the workgroups' shares of votes
// stay even.  Round r deals the slices G r .. G r + G - 1, slice G r + c to
// workgroup c, or with a rotation rot > 0 (G = 256, whole rounds) slice
// G r + ((b + rot r) mod G) to workgroup b, which moves a workgroup's slices
// across the columns of the frame from round to round.  The pixels outside the list
// get their final outputs here.  The launch also clears `hnext`, the
// histograms of the next frame.
struct FusedArgs {
    const void *fg;              // foreground plane (element type of the embedding), or null: every pixel
    float fg_thr;
    int32_t slice, seg_cap, rot;
    int32_t *list, *counts;
    int32_t *labels;
    float *score;
    unsigned long long *hnext;
    int32_t nnext;
};

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
// histograms `hrep` (clear when the frame starts: an earlier launch cleared
// them); the assignment launch that follows sums them and extracts the
// peaks.  Workgroup 0 also resets the pixel counts of the centroid records,
// which the assignment launch accumulates.
// MULTI: grids above 32 x 32 bins (one pass per block of 32 x 32 bins);
// otherwise the single block is compiled without the pass loop, whose
// registers would otherwise spill.  FUSED: the launch lists the
// participating pixels itself (FusedArgs); list and counts are then unused.
template <typename T, int F, bool MULTI, bool FUSED>
__global__ __launch_bounds__((kVoteWpb<T, F> * 64)) __attribute__((amdgpu_waves_per_eu(kVoteWaves<T, F>))) void k_vote_mfma(
    const T *__restrict__ emb, int32_t dstride, int32_t yoff, const int32_t *__restrict__ list,
    const int32_t *__restrict__ counts, int32_t nslices, int32_t slice_px, int32_t npix, Tables tb, int32_t Bw,
    int32_t Bh, unsigned long long *__restrict__ hrep,
    cpe_centroid *__restrict__ cents, int32_t cap, FusedArgs fz)
{
    static_assert(!(MULTI && FUSED), "the folded compaction serves single-block grids");
    constexpr int kWpb = kVoteWpb<T, F>;
    // blocks of 32 x 32 bins: one pass over the workgroup's tiles per block
    const int nbx = MULTI ? (Bw + kMfmaBins - 1) / kMfmaBins : 1, nby = MULTI ? (Bh + kMfmaBins - 1) / kMfmaBins : 1;
    // All LDS is static, so that table addresses are compile-time constants.
    __shared__ __align__(16) unsigned char smem[kVoteLds(kWpb, FUSED)];
    uint32_t *s_wt = reinterpret_cast<uint32_t *>(smem);                              // [kWKeys] fp16 limb pairs
    unsigned long long *s_h = reinterpret_cast<unsigned long long *>(s_wt + kWKeys);  // [32][kHStride], b * kHStride + a
    uint32_t *s_pop = reinterpret_cast<uint32_t *>(s_h + kMfmaBins * kHStride);      // palette operands
    uint32_t *s_ini = s_pop + kPopBytes / 4;                                          // [kWpb][2][32]
    int *s_pref = reinterpret_cast<int *>(s_ini + kWpb * 64);                        // [kMaxSlices + 1]
    int *s_next = s_pref + kMaxSlices + 1;                                            // next tile of the run
    int *s_cnt = s_next + 1;                                                          // FUSED: [2] pixels listed (LDS, global)
    int *s_list = s_pref + kMaxSlices + 5;                                            // FUSED: [kFusedMaxSeg]

    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int g = lane >> 5, ln = lane & 31;
    SliceLoad sl;
    if (!FUSED && list) slice_load(counts, nslices, sl);
    // the bin constants of this lane's bin in the first block (loaded with
    // the tables, not after the barrier, where they would cost a memory round
    // trip of their own)
    uint32_t np1x = tb.np1_x[ln], np1y = tb.np1_y[ln];
    {
        constexpr int kThreads = kWpb * 64, kN = kWKeys / 4, kPer = (kN + kThreads - 1) / kThreads;
        u32x4 w[kPer];
#pragma unroll
        for (int k = 0; k < kPer; k++) {
            const int i = k * kThreads + tid;
            w[k] = reinterpret_cast<const u32x4 *>(tb.wt_pk)[i < kN ? i : 0];
        }
        if constexpr (FUSED) {
            // While the table loads are in flight, two lists of the
            // participating pixels: (a) the assignment's, of this workgroup's
            // range lo .. hi-1 of the frame, in global memory, with the other
            // pixels' final outputs; (b) the vote's own, of its slices b,
            // b + G, ..., in LDS.  Both in steps of 64 lanes x 8 consecutive
            // pixels (b: slice r of the workgroup, chunk of 8 o, from lane
            // chunk 64 k + lane = r * slice / 8 + o), one step per wave at a
            // time (the code stays short: a launch fetches it cold, and
            // unrolling three steps measured 1.3 us slower per 640 x 640
            // frame); LDS counters hand out the positions.
            if (tid == 0) s_cnt[0] = s_cnt[1] = 0;
            __syncthreads();
            const int G = gridDim.x, b = blockIdx.x;
            const T *fgp = static_cast<const T *>(fz.fg);
            const bool vec = fgp && ((uintptr_t)fgp & 15u) == 0;
            const int lo = b * fz.seg_cap, hi = lo + fz.seg_cap < npix ? lo + fz.seg_cap : npix;
            const int steps_a = hi > lo ? (hi - lo + 511) >> 9 : 0;
            const int nsl = (npix + fz.slice - 1) / fz.slice;
            const int mine = b < nsl ? (nsl - 1 - b) / G + 1 : 0;
            const int csh = __builtin_ctz(fz.slice) - 3;                // log2 of the 8-pixel chunks per slice
            const int steps = steps_a + ((mine << csh) + 63) / 64;
            int32_t *seg = fz.list + (size_t)lo;
            // first pixel and limit of this lane's 8 in step j
            auto place = [&](int j, int &p0, int &lim) {
                if (j < steps_a) {
                    p0 = lo + j * 512 + lane * 8;
                    lim = hi;
                } else {
                    const int c = (j - steps_a) * 64 + lane, r = c >> csh;
                    const int sb = fz.rot ? (b + fz.rot * r) & (kMaxSlices - 1) : b;   // rot: G = kMaxSlices
                    p0 = (sb + G * r) * fz.slice + ((c & ((1 << csh) - 1)) << 3);
                    lim = r < mine ? npix : 0;
                }
            };
            // the next step's foreground words are loaded before this step's
            // are used
            int pn = 0, limn = 0;
            Raw8<T> rn = {};
            if (wv < steps) {
                place(wv, pn, limn);
                rn = load8_raw<T>(fgp, pn, limn, vec);
            }
            for (int j = wv; j < steps; j += kWpb) {
                const bool in_a = j < steps_a;                          // wave-uniform
                const int p0 = pn, lim = limn;
                const Raw8<T> rc = rn;
                if (j + kWpb < steps) {
                    place(j + kWpb, pn, limn);
                    rn = load8_raw<T>(fgp, pn, limn, vec);
                }
                float v[8];
                load8_values<T>(fgp, p0, lim, vec, rc, v);
                uint32_t m = 0, valid = 0;
#pragma unroll
                for (int i = 0; i < 8; i++) {
                    const bool in = p0 + i < lim;
                    valid |= (in ? 1u : 0u) << i;
                    m |= (in && (!fgp || v[i] > fz.fg_thr) ? 1u : 0u) << i;   // a NaN never exceeds it
                }
                const int c = __popc(m), incl = wave_incl_sum(c);
                const int tot = __builtin_amdgcn_readlane(incl, 63);
                int base = 0;
                if (lane == 0 && tot) base = atomicAdd(&s_cnt[in_a ? 1 : 0], tot);
                int off = __builtin_amdgcn_readfirstlane(base) + incl - c;
                if (in_a) {
#pragma unroll
                    for (int i = 0; i < 8; i++)
                        if ((m >> i) & 1u) seg[off++] = p0 + i;         // off < hi - lo <= seg_cap
                    const uint32_t bg = valid & ~m;
                    if (bg == 0xffu) {
                        const int4 z = {0, 0, 0, 0};
                        reinterpret_cast<int4 *>(fz.labels + p0)[0] = z;     // labels: 16-byte aligned
                        reinterpret_cast<int4 *>(fz.labels + p0)[1] = z;
                    } else if (bg) {
#pragma unroll
                        for (int i = 0; i < 8; i++)
                            if ((bg >> i) & 1u) fz.labels[p0 + i] = 0;
                    }
                    if (fz.score && bg) {
#pragma unroll
                        for (int i = 0; i < 8; i++)
                            if ((bg >> i) & 1u) fz.score[p0 + i] = 0.0f;
                    }
                } else {
#pragma unroll
                    for (int i = 0; i < 8; i++)
                        if ((m >> i) & 1u) s_list[off++] = p0 + i;      // off < the slices' pixels <= kFusedMaxSeg
                }
            }
            for (int i = b * kThreads + tid; i < fz.nnext; i += G * kThreads) fz.hnext[i] = 0ull;
        }
#pragma unroll
        for (int k = 0; k < kPer; k++) {
            const int i = k * kThreads + tid;
            if (i < kN) reinterpret_cast<u32x4 *>(s_wt)[i] = w[k];
        }
        for (int i = tid; i < kMfmaBins * kHStride; i += kThreads) s_h[i] = 0ull;
        for (int i = tid; i < kPopBytes / 16; i += kThreads) reinterpret_cast<u32x4 *>(s_pop)[i] = pop_block(tb.pop, i, 0, 0);
        if (tid == 0) *s_next = 0;
        if (!FUSED && list) slice_scan(sl, nslices, s_pref);
    }
    __syncthreads();
    // the workgroup's run of tiles: a share of the list, or (FUSED) its own pixels
    const int n = FUSED ? *s_cnt : list ? s_pref[nslices] : npix, ntiles = (n + 31) >> 5;
    int t0, tend;
    if constexpr (FUSED) {
        t0 = 0;
        tend = ntiles;
        if (tid == 0) fz.counts[blockIdx.x] = s_cnt[1];
    } else {
        block_run(ntiles, blockIdx.x, gridDim.x, t0, tend);
    }

    // this wave's |X|^2 per axis: [0] x, [1] y, by pixel
    uint32_t *ini = s_ini + wv * 64;
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

    // Packed weight limbs of the 16 (pixel, bin) results of one axis: the
    // accumulators start at the pixels' |X|^2, and cb = |P|^2 + 1 of this
    // lane's bin completes S + 1, whose binary32 bits give the bucket.
    auto weights = [&](const i32x16 &hh, const i32x16 &mid, const i32x16 &ll, uint32_t cb, uint32_t (&e)[16]) {
#pragma unroll
        for (int r = 0; r < 16; r++) {
            const uint32_t s1 = assemble(hh[r], mid[r], ll[r], cb);
            e[r] = s_wt[(__float_as_uint((float)s1) >> 15) & (kWKeys - 1)];
        }
    };

    // One tile of up to 32 pixels (queue slot m = lane & 31) from prefetched
    // input; `next` reuses the input registers once they are converted.
    auto tile = [&](RawSlices<T, F> &raw, int nvalid, auto next) {
        int n2x = 0, n2y = 0;
        AxisOp<F> X, Y;
        raw.convert(0, X, n2x);
        raw.convert(1, Y, n2y);
        after_convert(X, Y, n2x, n2y);
        next();
        n2x += __shfl_xor(n2x, 32);
        n2y += __shfl_xor(n2y, 32);
        if (g == 0) {
            ini[ln] = (uint32_t)n2x;
            ini[32 + ln] = (uint32_t)n2y;
        }
        uint32_t ex[16], ey[16];
        {
            i32x4 P[kPopKinds];
#pragma unroll
            for (int k = 0; k < kPopKinds; k++) P[k] = palette_operand(s_pop, 0, k, lane);
            i32x16 hh, mid, ll;
            axis_products<F, true>(X, P, row_init(ini, g), hh, mid, ll);
            weights(hh, mid, ll, np1x, ex);
        }
        {
            i32x4 P[kPopKinds];
#pragma unroll
            for (int k = 0; k < kPopKinds; k++) P[k] = palette_operand(s_pop, 1, k, lane);
            i32x16 hh, mid, ll;
            axis_products<F, true>(Y, P, row_init(ini + 32, g), hh, mid, ll);
            weights(hh, mid, ll, np1y, ey);
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

    for (int blk = 0; blk < nbx * nby; blk++) {
        const int bx = blk % nbx, by = blk / nbx;
        if (MULTI && blk > 0) {
            // the next block: its palette operands and bin constants, a clear
            // histogram and tile counter (the previous pass has flushed)
            np1x = tb.np1_x[kMfmaBins * bx + ln];
            np1y = tb.np1_y[kMfmaBins * by + ln];
            for (int i = tid; i < kMfmaBins * kHStride; i += blockDim.x) s_h[i] = 0ull;
            for (int i = tid; i < kPopBytes / 16; i += blockDim.x)
                reinterpret_cast<u32x4 *>(s_pop)[i] = pop_block(tb.pop, i, bx, by);
            if (tid == 0) *s_next = 0;
            __syncthreads();
        }
        int t = t0 + wv;
        ListCursor cur_list;
        if (!FUSED) cur_list.start(list, s_pref, nslices, slice_px, t < tend ? 32 * t : 0);
        // lane m of tile tt: entry 32 tt + m, or the tile's first entry past the end
        auto pixel = [&](int tt) {
            const int e = 32 * tt + ln < n ? 32 * tt + ln : 32 * tt;
            if constexpr (FUSED)
                return s_list[e];
            else
                return cur_list.pixel(e);
        };
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
        ntile = 0;

        // one global atomic per bin of the block
        __syncthreads();
        const int nb = Bw * Bh;
        unsigned long long *dst = hrep + (size_t)(blockIdx.x % kReplicas) * nb;
        for (int i = tid; i < kMfmaBins * kMfmaBins; i += blockDim.x) {
            const int b = kMfmaBins * by + i / kMfmaBins, a = kMfmaBins * bx + i % kMfmaBins;
            const unsigned long long v = s_h[(i / kMfmaBins) * kHStride + i % kMfmaBins];
            if (a < Bw && b < Bh && v) atomicAdd(dst + b * Bw + a, v);
        }
        __syncthreads();
    }
    if (blockIdx.x == 0)
        for (int k = tid; k < cap; k += blockDim.x) cents[k].npix = 0;
}

// ---------------------------------------------------------------------------
// Pass 2: assignment + label write-out
// ---------------------------------------------------------------------------
// Waves per SIMD of the assignment kernel: four where the register
// allocation fits 128 registers without spilling (vector input slices and up
// to 9 harmonics, or fp16 with 16), three otherwise; one workgroup per
// compute unit.
template <typename T, int F>
constexpr int kAssignWaves = (F <= 9 || (sizeof(T) == 2 && F == 16)) ? 4 : 3;
template <typename T, int F>
constexpr int kAssignWpb = 4 * kAssignWaves<T, F>;

// LDS bytes of k_assign_mfma: palette operands, |P|^2 by bin and by slot,
// candidate batches, bin -> centroid table, counts, per wave x and y
// distances [32 slots][kKeyStride] (u32), then the peak-extraction state
// (the searches merge their lanes' partial results in a wave's y array once
// it is no longer read).  The summed vote histogram (32 x 32 slots, 8 KB) of the prologue
// shares its bytes with the first waves' distance arrays, which are written
// only after it is no longer read.
constexpr size_t kAssignLdsCore(int wpb)
{
    return (size_t)kPopBytes + 4 * kMfmaBins * 4 + (size_t)kMaxBatchLds * 20 + kMfmaBins * kMfmaBins * 2 +
           kMfmaBins * kMfmaBins * 4 + (size_t)wpb * 2 * kMfmaBins * kKeyStride * 4 + sizeof(PeakLds) +
           (kMaxSlices + 1) * 4 + 16;
}
constexpr size_t kAssignLds(int wpb) { return (kAssignLdsCore(wpb) + 15) & ~(size_t)15; }

// Every workgroup first sums the vote histograms `hcur` of the vote launch
// and extracts the peaks in LDS (identical in every workgroup); workgroup 0
// writes the centroid records (all fields but the pixel count), K and the
// summed histogram `hlast`.
//
// Then, per tile of 32 pixels, the distances of both axes for the candidate
// slots (palette entries of the slots' bins as the MFMA rows, so that each
// lane holds one pixel and 16 slots) go to LDS as binary32 bits, laid out
// [slot][kKeyStride] so that lane m finds pixel m's value of any slot at a
// fixed stride.
// The candidate search walks the batches of 4 columns of one row (see the
// search below).  A pixel is labelled iff its distance sum D (in units of
// 1/4096) is below tau4096 = 4096 tau (Eq8; +inf: every pixel).
template <typename T, int F, bool FAST>
__global__ __launch_bounds__((kAssignWpb<T, F> * 64)) __attribute__((amdgpu_waves_per_eu(kAssignWaves<T, F>))) void k_assign_mfma(
    const T *__restrict__ emb, int32_t dstride, int32_t yoff, const int32_t *__restrict__ list,
    const int32_t *__restrict__ counts, int32_t nslices, int32_t slice_px, int32_t npix, double tau4096, Tables tb,
    const unsigned long long *__restrict__ hcur, unsigned long long *__restrict__ hlast, int32_t Bw, int32_t Bh, long long cut, int32_t cap,
    cpe_centroid *__restrict__ cents, int32_t *__restrict__ num, int32_t *__restrict__ labels,
    float *__restrict__ score_map, int32_t force_exact)
{
    constexpr int kWpb2 = kAssignWpb<T, F>;
    constexpr int kThreads = kWpb2 * 64;
    static_assert(kThreads >= kPeakThreads, "the peak prologue takes two histogram slots per thread");
    static_assert(kAssignLds(kWpb2) <= 160 * 1024, "LDS of one compute unit");
    static_assert(kMfmaBins * kMfmaBins * 8 <= 2 * kMfmaBins * kKeyStride * 4, "the summed histogram fits in wave 0's arrays");
    // All LDS is static, so that table addresses are compile-time constants.
    __shared__ __align__(16) unsigned char smem[kAssignLds(kWpb2)];
    uint32_t *s_pop = reinterpret_cast<uint32_t *>(smem);                            // palette operands
    uint32_t *s_cb = s_pop + kPopBytes / 4;                                          // [2][32] |P|^2 by bin
    uint32_t *s_cbs = s_cb + 2 * kMfmaBins;                                           // [2][32] by slot
    u32x4 *s_bo = reinterpret_cast<u32x4 *>(s_cbs + 2 * kMfmaBins);                // [kMaxBatchLds]
    uint32_t *s_bh = reinterpret_cast<uint32_t *>(s_bo + kMaxBatchLds);             // [kMaxBatchLds]
    uint16_t *s_rank = reinterpret_cast<uint16_t *>(s_bh + kMaxBatchLds);           // [32 * 32]
    int32_t *s_cnt = reinterpret_cast<int32_t *>(s_rank + kMfmaBins * kMfmaBins);   // [1024]
    uint32_t *s_keys = reinterpret_cast<uint32_t *>(s_cnt + kMfmaBins * kMfmaBins); // [kWpb2][2][32][kKeyStride]
    PeakLds &pl = *reinterpret_cast<PeakLds *>(s_keys + kWpb2 * 2 * kMfmaBins * kKeyStride);
    int *s_pref = reinterpret_cast<int *>(&pl + 1);                                  // [kMaxSlices + 1]
    int *s_next = s_pref + kMaxSlices + 1;                                            // next tile of the run
    unsigned long long *s_h = reinterpret_cast<unsigned long long *>(s_keys);              // [32 * 32] summed votes

    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const int g = lane >> 5, ln = lane & 31;
    const int nb = Bw * Bh;

    PeakLoad pld;                                   // issued before the table staging
    peaks_lds_load(hcur, Bw, Bh, pld);
    // This wave's search arrays, [slot][kKeyStride] per axis: x key of column
    // slot j, pixel m at kx[j * kKeyStride + m], y distance of row slot j at
    // ky[...].
    uint32_t *kx = s_keys + wv * 2 * kMfmaBins * kKeyStride;
    uint32_t *ky = kx + kMfmaBins * kKeyStride;
    SliceLoad sl;
    if (list) slice_load(counts, nslices, sl);
    for (int i = tid; i < kPopBytes / 16; i += kThreads) reinterpret_cast<u32x4 *>(s_pop)[i] = pop_block(tb.pop, i, 0, 0);
    if (tid < 2 * kMfmaBins) {
        const int bin = tid & (kMfmaBins - 1);
        s_cb[tid] = tid < kMfmaBins ? (bin < Bw ? tb.n2_x[bin] : 0u) : (bin < Bh ? tb.n2_y[bin] : 0u);
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
    __syncthreads();        // s_h is read; its bytes become distance arrays

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
    // bin, gathered once and kept in registers for the whole run; distances
    // are computed only for the groups of 8 slots that hold candidates.
    const int nslot[2] = {__builtin_amdgcn_readfirstlane(pl.ncol), __builtin_amdgcn_readfirstlane(pl.nrow)};
    // (the fast kernel reads them from LDS per tile: its search needs the
    // registers)
    const int slotbin[2] = {g * 32 + pl.colbin[ln], g * 32 + pl.rowbin[ln]};
    i32x4 popr[2][kPopKinds];
    if constexpr (!FAST) {
#pragma unroll
        for (int ax = 0; ax < 2; ax++)
#pragma unroll
            for (int k = 0; k < kPopKinds; k++) popr[ax][k] = palette_operand(s_pop, ax, k, slotbin[ax]);
    }

    // Distances of one tile (pixel m = lane & 31; this lane's 16 slots
    // acc_row(r, g) of each axis); `next` reuses the input registers once
    // they are converted.  The accumulators of the Xl.lo products start at
    // the slots' |P|^2; the pixel's |X|^2 completes S.  EXACT: the correctly
    // rounded square root of fl32(S); otherwise the hardware square root,
    // within one binary32 step of it (the fast search below).
    auto distances = [&](auto exact, RawSlices<T, F> &raw, auto next) {
        int n2x = 0, n2y = 0;
        AxisOp<F> X, Y;
        raw.convert(0, X, n2x);
        raw.convert(1, Y, n2y);
        after_convert(X, Y, n2x, n2y);
        next();
        const uint32_t npx = (uint32_t)(n2x + __shfl_xor(n2x, 32));
        const uint32_t npy = (uint32_t)(n2y + __shfl_xor(n2y, 32));
#pragma unroll
        for (int ax = 0; ax < 2; ax++) {
            i32x16 hh, mid, ll;
            i32x4 pop[kPopKinds];
#pragma unroll
            for (int k = 0; k < kPopKinds; k++) pop[k] = FAST ? palette_operand(s_pop, ax, k, slotbin[ax]) : popr[ax][k];
            axis_products<F, false>(ax ? Y : X, pop, row_init(s_cbs + ax * kMfmaBins, g), hh, mid, ll);
            const uint32_t np = ax ? npy : npx;
            uint32_t *dst = (ax ? ky : kx) + 4 * g * kKeyStride + ln;
#pragma unroll
            for (int r4 = 0; r4 < 4; r4++) {
                if (8 * r4 >= nslot[ax]) break;      // wave-uniform: no candidate in slots 8 r4 ..
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const int r = 4 * r4 + i;
                    const float x = (float)assemble(hh[r], mid[r], ll[r], np);
                    const float d = decltype(exact)::value ? sqrt_cr(x) : __builtin_amdgcn_sqrtf(x);
                    dst[kKeyStride * (8 * r4 + i)] = __float_as_uint(d);
                }
            }
        }
    };

    // Candidate search.  Lane l serves the four pixels 4 q .. 4 q + 3
    // (q = l & 7) for the batches j, j + 8, ... (j = l >> 3): one 16-byte
    // read fetches a column's distances of its four pixels, so each address
    // computation and each read serve four pixels.  Per batch and pixel the
    // smallest of the 4 x distances plus the row's y distance, summed exactly
    // in binary64, has at least 12 zero bits at the bottom of its mantissa
    // (both distances are 0 or binary32 values of at least 1, so the sum is a
    // multiple of 2^-23 below 2^17), which take the batch index (< 128).  The
    // eight lanes of a pixel quad then combine their minima through LDS; lane
    // m takes pixel m's result, finds the first column of the winning batch
    // with the batch's smallest x distance, and (lanes of half 0, valid
    // pixels) writes its label.
    auto search = [&](int pix, int nvalid) {
        __builtin_amdgcn_wave_barrier();
        const int q = lane & 7, j0 = lane >> 3;
        const unsigned char *kxq = reinterpret_cast<const unsigned char *>(kx + 4 * q);
        const unsigned char *kyq = reinterpret_cast<const unsigned char *>(ky + 4 * q);
        double b4[4] = {__builtin_inf(), __builtin_inf(), __builtin_inf(), __builtin_inf()};
        u32x4 o = s_bo[j0];                         // j0 < 8 <= nbat
        uint32_t hb = s_bh[j0];
        for (int bi = j0; bi < nbat; bi += 8) {     // nbat is a multiple of 8: the same count for every lane
            const u32x4 v0 = *reinterpret_cast<const u32x4 *>(kxq + o.x);
            const u32x4 v1 = *reinterpret_cast<const u32x4 *>(kxq + o.y);
            const u32x4 v2 = *reinterpret_cast<const u32x4 *>(kxq + o.z);
            const u32x4 v3 = *reinterpret_cast<const u32x4 *>(kxq + o.w);
            const u32x4 yd = *reinterpret_cast<const u32x4 *>(kyq + hb);
            if (bi + 8 < nbat) {                    // the next batch's offsets, read ahead
                o = s_bo[bi + 8];
                hb = s_bh[bi + 8];
            }
#pragma unroll
            for (int e = 0; e < 4; e++) {
                const uint32_t m = min(min(v0[e], v1[e]), min(v2[e], v3[e]));
                const double sum = (double)__uint_as_float(m) + (double)__uint_as_float(yd[e]);
                const unsigned long long sb = (unsigned long long)__double_as_longlong(sum);
                const unsigned long long key = (sb & ~0xffffffffull) | ((uint32_t)sb | (uint32_t)bi);
                b4[e] = min_f64(b4[e], __longlong_as_double((long long)key));
            }
        }
        // the eight lanes of a pixel quad combine through LDS (the y array
        // is no longer read): pixel m's partial key j at double 9 m + j (an
        // odd pixel stride spreads the banks); half g of the wave takes
        // j = 4g .. 4g + 3 for pixel m = lane & 31, then the halves exchange
        __builtin_amdgcn_wave_barrier();
        double *part = reinterpret_cast<double *>(ky);
#pragma unroll
        for (int e = 0; e < 4; e++) part[(4 * q + e) * 9 + j0] = b4[e];
        __builtin_amdgcn_wave_barrier();
        double bm = part[ln * 9 + 4 * g];
#pragma unroll
        for (int jj = 1; jj < 4; jj++) bm = min_f64(bm, part[ln * 9 + 4 * g + jj]);
        bm = min_f64(bm, __shfl_xor(bm, 32));
        __builtin_amdgcn_wave_barrier();
        const unsigned long long best = (unsigned long long)__double_as_longlong(bm);
        const int bi = (int)((uint32_t)best & 127u);
        const double D = __longlong_as_double((long long)(best & ~127ull));
        const u32x4 ow = s_bo[bi];
        const unsigned char *kxl = reinterpret_cast<const unsigned char *>(kx + ln);
        const uint32_t w0 = *reinterpret_cast<const uint32_t *>(kxl + ow.x);
        const uint32_t w1 = *reinterpret_cast<const uint32_t *>(kxl + ow.y);
        const uint32_t w2 = *reinterpret_cast<const uint32_t *>(kxl + ow.z);
        const uint32_t w3 = *reinterpret_cast<const uint32_t *>(kxl + ow.w);
        const uint32_t wm = min(min(w0, w1), min(w2, w3));
        const uint32_t col = (w0 == wm ? ow.x : w1 == wm ? ow.y : w2 == wm ? ow.z : ow.w) >> 7;   // column slot
        const uint32_t row = s_bh[bi] >> 7;                                                      // row slot
        if (g == 0 && ln < nvalid) {
            if (D < tau4096) {      // Eq8
                const int a = pl.colbin[col], b = pl.rowbin[row];
                const int k = s_rank[b * kMfmaBins + a] & (kMfmaBins * kMfmaBins - 1);
                labels[pix] = k + 1;
                if (score_map) score_map[pix] = expf(-(float)(D * 0x1p-12));
                atomicAdd(s_cnt + k, 1);
            } else {
                labels[pix] = 0;
                if (score_map) score_map[pix] = 0.0f;
            }
        }
        __builtin_amdgcn_wave_barrier();
    };

    // Fast search (labels only: no score map, tau = +inf).  The distances
    // are the hardware square roots r~ of fl32(S), each within one binary32
    // step of the correctly rounded r (cpe_check_sqrt verifies the step
    // correction of sqrt_cr, which only tries r~ and its two neighbours, on
    // every input).  Lane l serves the pixels 4q .. 4q + 3 (q = l & 7) over
    // the batches j, j + 8, ... (j = l >> 3) of the unpadded list, so that no
    // batch is seen twice (one 16-byte read fetches a column's distances of
    // its four pixels; the next batch's offsets are read ahead), and keeps
    // per pixel the smallest binary32 sum fl(min x~ + y~) of a batch, its
    // batch, and the second smallest.  A step at v is at most 2^-23 v, so
    // x~ + y~ lies within relative 2^-23 of x + y and the rounded sum s
    // within relative g = 3 2^-24 + 2^-47 of the batch's true minimum D.
    // If the second smallest sum exceeds the smallest s_w by kFastGap steps
    // (each more than 2^-24 s_w), so by more than 2g / (1 - g) s_w, every
    // other batch's D exceeds the winning batch's (a sum of 0 is exact: any
    // other distance sum is at least 1).
    // Within the winning batch (one row, exact distances of one y), a column
    // whose r~ is at least 3 steps above the batch's smallest r~ is strictly
    // farther.  When both hold the winner is the unique minimiser of the
    // exact sums, i.e. the candidate the exact search selects.  Otherwise
    // (near ties, within a few units in the last place) the wave recomputes
    // the tile exactly; false is returned and nothing is written.
    const int nbr = min(pl.nbat_real, kMaxBatchLds);
    auto search_fast = [&](int pix, int nvalid) -> bool {
        __builtin_amdgcn_wave_barrier();
        int lo = lane;
        __asm__ volatile("" : "+v"(lo));        // recomputed per tile, not held across the loop
        const int q = lo & 7, j0 = lo >> 3;
        const unsigned char *kxq = reinterpret_cast<const unsigned char *>(kx + 4 * q);
        const unsigned char *kyq = reinterpret_cast<const unsigned char *>(ky + 4 * q);
        float b[4], s2[4];
        int bx[4];
#pragma unroll
        for (int e = 0; e < 4; e++) {
            b[e] = s2[e] = __builtin_inff();
            bx[e] = 0;
        }
        u32x4 o = {};
        uint32_t hb = 0;
        if (j0 < nbr) {
            o = s_bo[j0];
            hb = s_bh[j0];
        }
        for (int bi = j0; bi < nbr; bi += 8) {
            const u32x4 v0 = *reinterpret_cast<const u32x4 *>(kxq + o.x);
            const u32x4 v1 = *reinterpret_cast<const u32x4 *>(kxq + o.y);
            const u32x4 v2 = *reinterpret_cast<const u32x4 *>(kxq + o.z);
            const u32x4 v3 = *reinterpret_cast<const u32x4 *>(kxq + o.w);
            const u32x4 yd = *reinterpret_cast<const u32x4 *>(kyq + hb);
            if (bi + 8 < nbr) {             // the next batch's offsets, read ahead
                o = s_bo[bi + 8];
                hb = s_bh[bi + 8];
            }
#pragma unroll
            for (int e = 0; e < 4; e++) {
                const uint32_t m = min(min(v0[e], v1[e]), min(v2[e], v3[e]));
                const float sm = __uint_as_float(m) + __uint_as_float(yd[e]);
                s2[e] = __builtin_amdgcn_fmed3f(b[e], s2[e], sm);
                bx[e] = sm < b[e] ? bi : bx[e];
                b[e] = sm < b[e] ? sm : b[e];
            }
        }
        // the eight lanes of a pixel quad combine through LDS (the y array
        // is no longer read): pixel m's partial j (smallest, second, batch)
        // at word 25 m + 3 j (an odd pixel stride spreads the banks); half g
        // of the wave merges j = 4g .. 4g + 3 for pixel m = lane & 31, then
        // the two halves exchange (as bit patterns, which order like the
        // non-negative sums; equal smallest sums leave a second smallest
        // equal to the smallest)
        __builtin_amdgcn_wave_barrier();
        uint32_t *part = ky;
#pragma unroll
        for (int e = 0; e < 4; e++) {
            uint32_t *w = part + (4 * q + e) * 25 + 3 * j0;
            w[0] = __float_as_uint(b[e]);
            w[1] = __float_as_uint(s2[e]);
            w[2] = (uint32_t)bx[e];
        }
        __builtin_amdgcn_wave_barrier();
        uint32_t ub = 0xffffffffu, us = 0xffffffffu, ux = 0;
#pragma unroll
        for (int jj = 0; jj < 4; jj++) {
            const uint32_t *rp = part + ln * 25 + 3 * (4 * g + jj);
            const u32x4 r = {rp[0], rp[1], rp[2], 0u};
            us = min(min(us, r.y), max(ub, r.x));
            ux = r.x < ub ? r.z : ux;
            ub = min(ub, r.x);
        }
        {
            const uint32_t ob = __shfl_xor(ub, 32), os = __shfl_xor(us, 32), ox = __shfl_xor(ux, 32);
            us = min(min(us, os), max(ub, ob));
            ux = ob < ub ? ox : ux;
            ub = min(ub, ob);
        }
        __builtin_amdgcn_wave_barrier();
        const int bi = (int)ux;
        const u32x4 ow = s_bo[bi];
        const unsigned char *kxl = reinterpret_cast<const unsigned char *>(kx + ln);
        const uint32_t w0 = *reinterpret_cast<const uint32_t *>(kxl + ow.x);
        const uint32_t w1 = *reinterpret_cast<const uint32_t *>(kxl + ow.y);
        const uint32_t w2 = *reinterpret_cast<const uint32_t *>(kxl + ow.z);
        const uint32_t w3 = *reinterpret_cast<const uint32_t *>(kxl + ow.w);
        const uint32_t wm = min(min(w0, w1), min(w2, w3));
        const uint32_t oc = w0 == wm ? ow.x : w1 == wm ? ow.y : w2 == wm ? ow.z : ow.w;   // first column at the minimum
        const bool near = (ow.x != oc && w0 - wm < 3u) || (ow.y != oc && w1 - wm < 3u) ||
                          (ow.z != oc && w2 - wm < 3u) || (ow.w != oc && w3 - wm < 3u);
        const bool amb = near || us - ub < (uint32_t)kFastGap;
        const bool valid = g == 0 && ln < nvalid;
        if (force_exact || __ballot(amb && valid)) return false;
        if (valid) {
            const int a = pl.colbin[oc >> 7], bb_ = pl.rowbin[s_bh[bi] >> 7];
            const int k = s_rank[bb_ * kMfmaBins + a] & (kMfmaBins * kMfmaBins - 1);
            labels[pix] = k + 1;
            atomicAdd(s_cnt + k, 1);
        }
        __builtin_amdgcn_wave_barrier();
        return true;
    };

    // Exact search of the tiles the fast search leaves undecided: lane m
    // (either half: half g takes the batches g, g + 2, ...) scans every batch
    // for pixel m with the keys of the exact search above (binary64 sum of
    // the batch's smallest x distance and the row's y distance, batch index
    // in the low bits), then takes the first column of the winning batch at
    // the batch's minimum: the same candidate as the exact search.
    auto search_pix = [&](int pix, int nvalid) {
        __builtin_amdgcn_wave_barrier();
        const unsigned char *kxl = reinterpret_cast<const unsigned char *>(kx + ln);
        const unsigned char *kyl = reinterpret_cast<const unsigned char *>(ky + ln);
        double best = __builtin_inf();
        for (int bi = g; bi < nbr; bi += 2) {
            const u32x4 o = s_bo[bi];
            const uint32_t w0 = *reinterpret_cast<const uint32_t *>(kxl + o.x);
            const uint32_t w1 = *reinterpret_cast<const uint32_t *>(kxl + o.y);
            const uint32_t w2 = *reinterpret_cast<const uint32_t *>(kxl + o.z);
            const uint32_t w3 = *reinterpret_cast<const uint32_t *>(kxl + o.w);
            const uint32_t yv = *reinterpret_cast<const uint32_t *>(kyl + s_bh[bi]);
            const uint32_t m = min(min(w0, w1), min(w2, w3));
            const double sum = (double)__uint_as_float(m) + (double)__uint_as_float(yv);
            const unsigned long long sb = (unsigned long long)__double_as_longlong(sum);
            best = min_f64(best, __longlong_as_double((long long)((sb & ~0xffffffffull) | ((uint32_t)sb | (uint32_t)bi))));
        }
        best = min_f64(best, __shfl_xor(best, 32));
        const int bi = (int)((uint32_t)__double_as_longlong(best) & 127u);
        const u32x4 o = s_bo[bi];
        const uint32_t w0 = *reinterpret_cast<const uint32_t *>(kxl + o.x);
        const uint32_t w1 = *reinterpret_cast<const uint32_t *>(kxl + o.y);
        const uint32_t w2 = *reinterpret_cast<const uint32_t *>(kxl + o.z);
        const uint32_t w3 = *reinterpret_cast<const uint32_t *>(kxl + o.w);
        const uint32_t wm = min(min(w0, w1), min(w2, w3));
        const uint32_t col = (w0 == wm ? o.x : w1 == wm ? o.y : w2 == wm ? o.z : o.w) >> 7;
        if (g == 0 && ln < nvalid) {
            const int a = pl.colbin[col], b = pl.rowbin[s_bh[bi] >> 7];
            const int k = s_rank[b * kMfmaBins + a] & (kMfmaBins * kMfmaBins - 1);
            labels[pix] = k + 1;
            atomicAdd(s_cnt + k, 1);
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
        auto next = [&]() {
            if (tn < tend) {
                raw.load(emb + (size_t)ipn * dstride, yoff, g);
                tnn = take_tile(s_next, lane, t0, kWpb2);
                if (tnn < tend) ipnn = pixel(tnn);
            }
        };
        const int nvalid = min(32, n - 32 * t);
        if constexpr (FAST) {
            distances(std::false_type{}, raw, next);
            if (!search_fast(ip, nvalid)) {
                raw.load(emb + (size_t)ip * dstride, yoff, g);          // this tile's rows again
                distances(std::true_type{}, raw, []() {});
                if (tn < tend) raw.load(emb + (size_t)ipn * dstride, yoff, g);   // the next tile's rows again
                search_pix(ip, nvalid);
            }
        } else {
            distances(std::true_type{}, raw, next);
            search(ip, nvalid);
        }
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
