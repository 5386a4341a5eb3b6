// cpe_decode.hip -- gfx950 decoder for sinusoidal centroid encodings.
//
// Host side: argument checking, construction of the Eq9 palettes and the
// weight table in fp64 (once, at create), one device allocation for all
// constants and scratch, and the launch sequence of cpe_decode.
//
// Device side, three launches per frame on the caller's stream:
//   k_vote    per-pixel centroid recovery (Eq4/Eq10: distances of the
//             pixel's x^ and y^ to every palette entry, weights e^-d from
//             the table) and soft voting (Eq6/Eq11) into a block-private
//             register-tiled 64-bit histogram, flushed with global atomics
//             into one of kReplicas replicated histograms;
//   k_peaks   one workgroup: sums the replicas (and clears them for the next
//             frame), finds strict 8-neighbour local maxima above the
//             threshold (local-maxima search, Section 3.2) and compacts
//             them in bin order with wave ballots and a prefix sum;
//   k_assign  nearest-candidate assignment (Eq7) of every foreground pixel,
//             label write-out, optional score map, per-centroid pixel counts
//             (mask aggregation, Section 3.2) privatised in LDS.
//
// The arithmetic is the fixed-point contract described in cpe_decode.h; all
// vote sums are exact integers, so the result does not depend on the order
// in which pixels, waves or blocks are processed.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

#include "cpe_decode.h"

namespace {

constexpr int kWMant = 8;                  // weight bucket: top 8 mantissa bits of fl32(S+1)
constexpr int kCMant = 9;                  // code bucket: top 9 mantissa bits
constexpr int kWKeys = 32 << kWMant;       // 8192 weight buckets
constexpr int kCKeys = 32 << kCMant;       // 16384 code buckets
constexpr int kReplicas = 16;       // replicated global histograms (atomic spread)
constexpr int kMaxF = 16;
constexpr int kMaxBins = 128;
constexpr int kCountCap = 1024;     // centroids whose counts are privatised in LDS

typedef short v2s __attribute__((ext_vector_type(2)));

struct Tables {
    const int32_t *pal_x;   // [Bw][F]: harmonic k = (sin | cos << 16), int16 each, x4096
    const int32_t *pal_y;   // [Bh][F]
    const uint32_t *n2_x;   // [Bw]  sum of squared palette entries
    const uint32_t *n2_y;   // [Bh]
    const uint16_t *wt;     // [kWKeys] 2^15 e^-d per 8-bit bucket
    const uint16_t *ct;     // [kCKeys] 4096 d per 9-bit bucket
    const float *cx;        // [Bw] bin centres (pixels)
    const float *cy;        // [Bh]
};

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

}  // namespace

struct cpe_decoder {
    int32_t H, W, D, F, bins_w, bins_h, cap;
    cpe_dtype dtype;
    int device;
    std::vector<int16_t> pal_x, pal_y;   // host copies, [bins][2F]
    std::vector<uint16_t> wt, ct;        // host copies of the bucket tables
    unsigned char *dev;                  // single device allocation
    size_t dev_bytes;
    Tables tb;
    unsigned long long *hrep;            // [kReplicas][nb]
    unsigned long long *hlast;           // [nb]
    int32_t *peaks;                      // [cap] a | b << 16
    int32_t *kinfo;                      // [0] = min(K, cap), [1] = K
    hipEvent_t stage_ev[CPE_STAGE_EVENTS];
    bool stage_on;
};

// ---------------------------------------------------------------------------
// device helpers
// ---------------------------------------------------------------------------
namespace {

// Input to fixed point: rint(4096 clamp(v, -1.5, 1.5)); a NaN clamps to -1.5.
__device__ __forceinline__ int32_t to_fixed(float v)
{
    const float c = fminf(fmaxf(v, -1.5f), 1.5f);   // maxnum/minnum: NaN -> -1.5
    return (int32_t)rintf(c * 4096.0f);
}

__device__ __forceinline__ int32_t pack2(int32_t lo, int32_t hi)
{
    return (int32_t)(((uint32_t)lo & 0xffffu) | ((uint32_t)hi << 16));
}

__device__ __forceinline__ float half_bits_to_float(uint32_t bits)
{
    return (float)__builtin_bit_cast(_Float16, (uint16_t)bits);
}

template <typename T> __device__ __forceinline__ float load_scalar(const T *p);
template <> __device__ __forceinline__ float load_scalar<float>(const float *p) { return *p; }
template <> __device__ __forceinline__ float load_scalar<_Float16>(const _Float16 *p) { return (float)*p; }

// Load one axis block (2F channels) of a pixel and pack it as F int16 pairs.
template <typename T, int F, int ALIGN>
__device__ __forceinline__ void load_block(const T *blk, int32_t (&pk)[F])
{
    if constexpr (sizeof(T) == 4) {
        const float *p = reinterpret_cast<const float *>(__builtin_assume_aligned(blk, ALIGN));
#pragma unroll
        for (int k = 0; k < F; k++) pk[k] = pack2(to_fixed(p[2 * k]), to_fixed(p[2 * k + 1]));
    } else {
        const uint32_t *p = reinterpret_cast<const uint32_t *>(__builtin_assume_aligned(blk, ALIGN));
#pragma unroll
        for (int k = 0; k < F; k++) {
            uint32_t w = p[k];
            pk[k] = pack2(to_fixed(half_bits_to_float(w & 0xffffu)), to_fixed(half_bits_to_float(w >> 16)));
        }
    }
}

template <int F>
__device__ __forceinline__ int32_t dot_pk(const int32_t (&x)[F], const int32_t *p)
{
    int32_t acc = 0;
#pragma unroll
    for (int k = 0; k < F; k++)
        acc = __builtin_amdgcn_sdot2(__builtin_bit_cast(v2s, x[k]), __builtin_bit_cast(v2s, p[k]), acc, false);
    return acc;
}

// S = |X|^2 + |P|^2 - 2 X.P is exact modulo 2^32 and lies in [0, 2^32).
__device__ __forceinline__ uint32_t axis_s(uint32_t nX, uint32_t nP, int32_t dot)
{
    return nX + nP - 2u * (uint32_t)dot;
}

// m-bit distance bucket: exponent and top m mantissa bits of fl32(S+1).
template <int M>
__device__ __forceinline__ int dist_key(uint32_t s)
{
    const uint32_t bits = __float_as_uint((float)(s + 1u));
    return (int)(bits >> (23 - M)) - (127 << M);
}

template <typename T, int F>
struct PixelLayout {
    static constexpr int kRowBytes = 4 * F * (int)sizeof(T);
    static constexpr int kAlignX = (kRowBytes % 16 == 0) ? 16 : 4;
    static constexpr int kAlignY = (kAlignX == 16 && (2 * F * (int)sizeof(T)) % 16 == 0) ? 16 : 4;
};

// ---------------------------------------------------------------------------
// S1 + S2: recovery and soft voting
// ---------------------------------------------------------------------------
template <typename T, int F>
__global__ __launch_bounds__(256) void k_vote(const T *__restrict__ emb, const T *__restrict__ fg, int32_t npix,
                                              float fg_thr, Tables tb, int32_t Bw, int32_t Bh,
                                              unsigned long long *__restrict__ hrep)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int TP = blockDim.x;
    const int tid = threadIdx.x;
    int32_t *s_px = reinterpret_cast<int32_t *>(smem);
    int32_t *s_py = s_px + Bw * F;
    uint32_t *s_nx = reinterpret_cast<uint32_t *>(s_py + Bh * F);
    uint32_t *s_ny = s_nx + Bw;
    int32_t *s_list = reinterpret_cast<int32_t *>(s_ny + Bh);   // [TP]
    int32_t *s_n = s_list + TP;                                  // [4]
    uint16_t *s_wt = reinterpret_cast<uint16_t *>(s_n + 4);      // [kWKeys]
    uint16_t *s_qx = s_wt + kWKeys;                              // [Bw][TP]
    uint16_t *s_qy = s_qx + Bw * TP;                             // [Bh][TP]

    for (int i = tid; i < Bw * F; i += TP) s_px[i] = tb.pal_x[i];
    for (int i = tid; i < Bh * F; i += TP) s_py[i] = tb.pal_y[i];
    for (int i = tid; i < Bw; i += TP) s_nx[i] = tb.n2_x[i];
    for (int i = tid; i < Bh; i += TP) s_ny[i] = tb.n2_y[i];
    for (int i = tid; i < kWKeys; i += TP) s_wt[i] = tb.wt[i];

    using L = PixelLayout<T, F>;
    const int nb = Bw * Bh;
    const int per_chunk = 4 * TP;
    const int nchunks = (nb + per_chunk - 1) / per_chunk;
    unsigned long long *hdst = hrep + (size_t)(blockIdx.x % kReplicas) * nb;

    unsigned long long acc[4] = {0ull, 0ull, 0ull, 0ull};
    int ba[4], bb[4];
#pragma unroll
    for (int j = 0; j < 4; j++) {
        int bin = j * TP + tid;
        ba[j] = bin % Bw;
        bb[j] = (bin / Bw) < Bh ? bin / Bw : 0;
    }

    for (int64_t tile = blockIdx.x; tile * TP < npix; tile += gridDim.x) {
        if (tid == 0) *s_n = 0;
        __syncthreads();
        const int64_t p = tile * TP + tid;
        if (p < npix && load_scalar<T>(fg + p) > fg_thr) {
            int slot = atomicAdd(s_n, 1);
            s_list[slot] = (int32_t)p;
        }
        __syncthreads();
        const int n = *s_n;
        if (tid < n) {
            const T *row = emb + (size_t)s_list[tid] * (4 * F);
            int32_t xk[F], yk[F];
            load_block<T, F, L::kAlignX>(row, xk);
            load_block<T, F, L::kAlignY>(row + 2 * F, yk);
            const uint32_t nX = (uint32_t)dot_pk<F>(xk, xk);
            const uint32_t nY = (uint32_t)dot_pk<F>(yk, yk);
            for (int a = 0; a < Bw; a++)
                s_qx[a * TP + tid] = s_wt[dist_key<kWMant>(axis_s(nX, s_nx[a], dot_pk<F>(xk, s_px + a * F)))];
            for (int b = 0; b < Bh; b++)
                s_qy[b * TP + tid] = s_wt[dist_key<kWMant>(axis_s(nY, s_ny[b], dot_pk<F>(yk, s_py + b * F)))];
        }
        __syncthreads();
        if (nchunks == 1) {
            for (int i = 0; i < n; i++) {
#pragma unroll
                for (int j = 0; j < 4; j++)
                    acc[j] += (unsigned long long)((uint32_t)s_qx[ba[j] * TP + i] * (uint32_t)s_qy[bb[j] * TP + i]);
            }
        } else {
            for (int c = 0; c < nchunks; c++) {
                unsigned long long part[4] = {0ull, 0ull, 0ull, 0ull};
                int ca[4], cb[4];
#pragma unroll
                for (int j = 0; j < 4; j++) {
                    int bin = c * per_chunk + j * TP + tid;
                    ca[j] = bin % Bw;
                    cb[j] = (bin / Bw) < Bh ? bin / Bw : 0;
                }
                for (int i = 0; i < n; i++) {
#pragma unroll
                    for (int j = 0; j < 4; j++)
                        part[j] += (unsigned long long)((uint32_t)s_qx[ca[j] * TP + i] * (uint32_t)s_qy[cb[j] * TP + i]);
                }
#pragma unroll
                for (int j = 0; j < 4; j++) {
                    int bin = c * per_chunk + j * TP + tid;
                    if (bin < nb && part[j]) atomicAdd(hdst + bin, part[j]);
                }
            }
        }
        __syncthreads();
    }
    if (nchunks == 1) {
#pragma unroll
        for (int j = 0; j < 4; j++) {
            int bin = j * TP + tid;
            if (bin < nb && acc[j]) atomicAdd(hdst + bin, acc[j]);
        }
    }
}

// ---------------------------------------------------------------------------
// S3: peak extraction and compaction (one workgroup of 1024 threads)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void k_peaks(unsigned long long *__restrict__ hrep,
                                                unsigned long long *__restrict__ hlast, int32_t Bw, int32_t Bh,
                                                long long cut, int32_t cap, const float *__restrict__ cx,
                                                const float *__restrict__ cy, cpe_centroid *__restrict__ out,
                                                int32_t *__restrict__ num_out, int32_t *__restrict__ peaks,
                                                int32_t *__restrict__ kinfo)
{
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned long long *s_h = reinterpret_cast<unsigned long long *>(smem);   // [nb]
    __shared__ int s_wave[16];
    __shared__ int s_base;
    const int tid = threadIdx.x;
    const int nb = Bw * Bh;
    for (int i = tid; i < nb; i += blockDim.x) {
        unsigned long long s = 0;
        for (int r = 0; r < kReplicas; r++) {
            s += hrep[(size_t)r * nb + i];
            hrep[(size_t)r * nb + i] = 0ull;
        }
        s_h[i] = s;
        hlast[i] = s;
    }
    if (tid == 0) s_base = 0;
    __syncthreads();

    const int lane = tid & 63, wid = tid >> 6, nwaves = blockDim.x >> 6;
    for (int c0 = 0; c0 < nb; c0 += blockDim.x) {
        const int i = c0 + tid;
        bool flag = false;
        int a = 0, b = 0;
        unsigned long long v = 0;
        if (i < nb) {
            a = i % Bw;
            b = i / Bw;
            v = s_h[i];
            flag = (long long)v > cut;
            for (int db = -1; db <= 1; db++)
                for (int da = -1; da <= 1; da++) {
                    if (!da && !db) continue;
                    const int nb_ = b + db, na = a + da;
                    if (nb_ < 0 || nb_ >= Bh || na < 0 || na >= Bw) continue;
                    if (!(v > s_h[nb_ * Bw + na])) flag = false;
                }
        }
        const unsigned long long mask = __ballot(flag);
        const int before = __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0));
        if (lane == 0) s_wave[wid] = __popcll(mask);
        __syncthreads();
        int off = s_base;
        for (int w = 0; w < wid; w++) off += s_wave[w];
        if (flag) {
            const int pos = off + before;
            if (pos < cap) {
                cpe_centroid rec;
                rec.bin_x = a;
                rec.bin_y = b;
                rec.x = cx[a];
                rec.y = cy[b];
                rec.score = (double)v * 0x1p-30;
                rec.npix = 0;
                rec.reserved = 0;
                out[pos] = rec;
                peaks[pos] = a | (b << 16);
            }
        }
        __syncthreads();
        if (tid == 0) {
            int tot = 0;
            for (int w = 0; w < nwaves; w++) tot += s_wave[w];
            s_base += tot;
        }
        __syncthreads();
    }
    if (tid == 0) {
        *num_out = s_base;
        kinfo[0] = s_base < cap ? s_base : cap;
        kinfo[1] = s_base;
    }
}

// ---------------------------------------------------------------------------
// S4 + S5: assignment, label write-out, counts
// ---------------------------------------------------------------------------
template <typename T, int F>
__global__ __launch_bounds__(256) void k_assign(const T *__restrict__ emb, const T *__restrict__ fg, int32_t npix,
                                                float fg_thr, Tables tb, int32_t Bw, int32_t Bh,
                                                const int32_t *__restrict__ peaks, const int32_t *__restrict__ kinfo,
                                                cpe_centroid *__restrict__ cents, int32_t *__restrict__ labels,
                                                float *__restrict__ score_map)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int TP = blockDim.x;
    const int tid = threadIdx.x;
    int32_t *s_px = reinterpret_cast<int32_t *>(smem);
    int32_t *s_py = s_px + Bw * F;
    uint32_t *s_nx = reinterpret_cast<uint32_t *>(s_py + Bh * F);
    uint32_t *s_ny = s_nx + Bw;
    int32_t *s_list = reinterpret_cast<int32_t *>(s_ny + Bh);   // [TP]
    int32_t *s_n = s_list + TP;                                  // [4]
    int32_t *s_cnt = s_n + 4;                                    // [kCountCap]
    int32_t *s_r = s_cnt + kCountCap;                            // [Bw + Bh][TP] codes
    uint16_t *s_ct = reinterpret_cast<uint16_t *>(s_r + (Bw + Bh) * TP);   // [kCKeys]

    const int Kc = kinfo[0];
    const int ncnt = Kc < kCountCap ? Kc : kCountCap;
    for (int i = tid; i < Bw * F; i += TP) s_px[i] = tb.pal_x[i];
    for (int i = tid; i < Bh * F; i += TP) s_py[i] = tb.pal_y[i];
    for (int i = tid; i < Bw; i += TP) s_nx[i] = tb.n2_x[i];
    for (int i = tid; i < Bh; i += TP) s_ny[i] = tb.n2_y[i];
    for (int i = tid; i < ncnt; i += TP) s_cnt[i] = 0;
    for (int i = tid; i < kCKeys; i += TP) s_ct[i] = tb.ct[i];

    using L = PixelLayout<T, F>;
    for (int64_t tile = blockIdx.x; tile * TP < npix; tile += gridDim.x) {
        if (tid == 0) *s_n = 0;
        __syncthreads();
        const int64_t p = tile * TP + tid;
        if (p < npix) {
            const bool part = Kc > 0 && load_scalar<T>(fg + p) > fg_thr;
            if (part) {
                int slot = atomicAdd(s_n, 1);
                s_list[slot] = (int32_t)p;
            } else {
                labels[p] = 0;
                if (score_map) score_map[p] = 0.0f;
            }
        }
        __syncthreads();
        const int n = *s_n;
        if (tid < n) {
            const int32_t pp = s_list[tid];
            const T *row = emb + (size_t)pp * (4 * F);
            int32_t xk[F], yk[F];
            load_block<T, F, L::kAlignX>(row, xk);
            load_block<T, F, L::kAlignY>(row + 2 * F, yk);
            const uint32_t nX = (uint32_t)dot_pk<F>(xk, xk);
            const uint32_t nY = (uint32_t)dot_pk<F>(yk, yk);
            for (int a = 0; a < Bw; a++)
                s_r[a * TP + tid] = s_ct[dist_key<kCMant>(axis_s(nX, s_nx[a], dot_pk<F>(xk, s_px + a * F)))];
            for (int b = 0; b < Bh; b++)
                s_r[(Bw + b) * TP + tid] = s_ct[dist_key<kCMant>(axis_s(nY, s_ny[b], dot_pk<F>(yk, s_py + b * F)))];
            int best = 0;
            const int32_t pk0 = peaks[0];
            int32_t bd = s_r[(pk0 & 0xffff) * TP + tid] + s_r[(Bw + (pk0 >> 16)) * TP + tid];
            for (int k = 1; k < Kc; k++) {
                const int32_t pk = peaks[k];
                const int32_t d = s_r[(pk & 0xffff) * TP + tid] + s_r[(Bw + (pk >> 16)) * TP + tid];
                if (d < bd) {
                    bd = d;
                    best = k;
                }
            }
            labels[pp] = best + 1;
            if (score_map) score_map[pp] = expf(-((float)bd * 0x1p-12f));
            if (best < kCountCap)
                atomicAdd(s_cnt + best, 1);
            else
                atomicAdd(&cents[best].npix, 1);
        }
        __syncthreads();
    }
    __syncthreads();
    for (int i = tid; i < ncnt; i += TP)
        if (s_cnt[i]) atomicAdd(&cents[i].npix, s_cnt[i]);
}

// ---------------------------------------------------------------------------
// launch helpers
// ---------------------------------------------------------------------------
// Largest pixel tile (threads per block) whose LDS footprint fits the budget.
int pick_tile(size_t fixed, size_t per_px, size_t budget)
{
    for (int tp = 256; tp >= 64; tp >>= 1)
        if (fixed + per_px * (size_t)tp <= budget) return tp;
    return 64;
}

template <typename T, int F>
cpe_status launch_all(cpe_decoder *h, hipStream_t stream, const void *emb, const void *fg, float fg_thr,
                      long long cut, cpe_centroid *cents, int32_t *num, int32_t *labels, float *score)
{
    const int Bw = h->bins_w, Bh = h->bins_h, nb = Bw * Bh;
    const int npix = h->H * h->W;
    const T *e = static_cast<const T *>(emb);
    const T *g = static_cast<const T *>(fg);
    auto mark = [&](int i) {
        if (h->stage_on) (void)hipEventRecord(h->stage_ev[i], stream);
    };
    mark(0);

    const size_t tables = (size_t)(Bw + Bh) * F * 4 + (size_t)(Bw + Bh) * 4;
    const size_t vote_fixed = tables + 16 + kWKeys * 2;
    const int tp1 = pick_tile(vote_fixed, (size_t)(Bw + Bh) * 2 + 4, 96 * 1024);
    const size_t lds1 = vote_fixed + (size_t)tp1 * 4 + (size_t)(Bw + Bh) * tp1 * 2;
    const int64_t tiles1 = ((int64_t)npix + tp1 - 1) / tp1;
    const int grid1 = (int)(tiles1 < 1024 ? tiles1 : 1024);
    hipLaunchKernelGGL((k_vote<T, F>), dim3(grid1), dim3(tp1), lds1, stream, e, g, npix, fg_thr, h->tb, Bw, Bh,
                       h->hrep);
    mark(1);

    hipLaunchKernelGGL(k_peaks, dim3(1), dim3(1024), (size_t)nb * 8, stream, h->hrep, h->hlast, Bw, Bh, cut, h->cap,
                       h->tb.cx, h->tb.cy, cents, num, h->peaks, h->kinfo);
    mark(2);

    const size_t asg_fixed = tables + 16 + kCountCap * 4 + kCKeys * 2;
    const int tp3 = pick_tile(asg_fixed, (size_t)(Bw + Bh) * 4 + 4, 120 * 1024);
    const size_t lds3 = asg_fixed + (size_t)tp3 * 4 + (size_t)(Bw + Bh) * tp3 * 4;
    const int64_t tiles3 = ((int64_t)npix + tp3 - 1) / tp3;
    const int grid3 = (int)(tiles3 < 2048 ? tiles3 : 2048);
    hipLaunchKernelGGL((k_assign<T, F>), dim3(grid3), dim3(tp3), lds3, stream, e, g, npix, fg_thr, h->tb, Bw, Bh,
                       h->peaks, h->kinfo, cents, labels, score);
    mark(3);
    return hipGetLastError() == hipSuccess ? CPE_OK : CPE_ERR_HIP;
}

template <typename T>
cpe_status dispatch_f(cpe_decoder *h, hipStream_t s, const void *emb, const void *fg, float thr, long long cut,
                      cpe_centroid *c, int32_t *n, int32_t *l, float *sc)
{
    switch (h->F) {
#define CPE_CASE(FF) \
    case FF:         \
        return launch_all<T, FF>(h, s, emb, fg, thr, cut, c, n, l, sc);
        CPE_CASE(1) CPE_CASE(2) CPE_CASE(3) CPE_CASE(4) CPE_CASE(5) CPE_CASE(6) CPE_CASE(7) CPE_CASE(8)
        CPE_CASE(9) CPE_CASE(10) CPE_CASE(11) CPE_CASE(12) CPE_CASE(13) CPE_CASE(14) CPE_CASE(15) CPE_CASE(16)
#undef CPE_CASE
    default:
        return CPE_ERR_UNSUPPORTED;
    }
}

long long peak_cut(double theta)
{
    const double t = std::floor(theta * 1073741824.0);
    if (t < -1.0) return -1;
    if (t > 4.0e18) return 4000000000000000000LL;
    return (long long)t;
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" {

const char *cpe_status_string(cpe_status s)
{
    switch (s) {
    case CPE_OK: return "ok";
    case CPE_ERR_INVALID_ARG: return "invalid argument";
    case CPE_ERR_UNSUPPORTED: return "unsupported configuration";
    case CPE_ERR_OUT_OF_MEMORY: return "out of device memory";
    case CPE_ERR_HIP: return "HIP runtime error";
    }
    return "unknown status";
}

cpe_status cpe_decode_create(cpe_decoder **out, int32_t H, int32_t W, int32_t D, cpe_dtype dtype,
                             const double *freq_x, const double *freq_y, int32_t n_freq, int32_t bins_w,
                             int32_t bins_h, int32_t centroid_capacity)
{
    if (!out) return CPE_ERR_INVALID_ARG;
    *out = nullptr;
    if (H < 1 || W < 1 || (int64_t)H * W > 2147483647LL) return CPE_ERR_INVALID_ARG;
    if (n_freq < 1 || n_freq > kMaxF || D != 4 * n_freq) return CPE_ERR_INVALID_ARG;
    if (dtype != CPE_F32 && dtype != CPE_F16) return CPE_ERR_INVALID_ARG;
    if (!freq_x || !freq_y) return CPE_ERR_INVALID_ARG;
    if (bins_w < 1 || bins_w > kMaxBins || bins_h < 1 || bins_h > kMaxBins) return CPE_ERR_INVALID_ARG;
    if (centroid_capacity < 1 || centroid_capacity > bins_w * bins_h) return CPE_ERR_INVALID_ARG;
    for (int k = 0; k < n_freq; k++)
        if (!std::isfinite(freq_x[k]) || !std::isfinite(freq_y[k])) return CPE_ERR_INVALID_ARG;

    cpe_decoder *h = new (std::nothrow) cpe_decoder();
    if (!h) return CPE_ERR_OUT_OF_MEMORY;
    h->H = H;
    h->W = W;
    h->D = D;
    h->F = n_freq;
    h->bins_w = bins_w;
    h->bins_h = bins_h;
    h->cap = centroid_capacity;
    h->dtype = dtype;
    if (hipGetDevice(&h->device) != hipSuccess) {
        delete h;
        return CPE_ERR_HIP;
    }
    const int F = n_freq, twoF = 2 * n_freq, nb = bins_w * bins_h;

    // Eq9 palettes: gamma at the bin centres (a+1) * extent / (n+1), x4096.
    auto palette = [&](int n, int extent, const double *freq, std::vector<int16_t> &pal, std::vector<float> &centres) {
        pal.assign((size_t)n * twoF, 0);
        centres.assign(n, 0.0f);
        for (int a = 0; a < n; a++) {
            const double c = ((double)(a + 1) * (double)extent) / (double)(n + 1);
            centres[a] = (float)c;
            for (int k = 0; k < F; k++) {
                const double ph = freq[k] * c;
                pal[(size_t)a * twoF + 2 * k] = (int16_t)std::rint(4096.0 * std::sin(ph));
                pal[(size_t)a * twoF + 2 * k + 1] = (int16_t)std::rint(4096.0 * std::cos(ph));
            }
        }
    };
    std::vector<float> cx, cy;
    palette(bins_w, W, freq_x, h->pal_x, cx);
    palette(bins_h, H, freq_y, h->pal_y, cy);
    // bucket tables: weight 2^15 e^-d (8-bit buckets), code 4096 d (9-bit
    // buckets), d taken at the bucket centre of fl32(S+1)
    auto centre_distance = [](int key, int m) {
        if (key == 0) return 0.0;
        const int e = key >> m, t = key & ((1 << m) - 1);
        return std::sqrt(std::ldexp(1.0 + ((double)t + 0.5) / (double)(1 << m), e) - 1.0) / 4096.0;
    };
    h->wt.resize(kWKeys);
    h->ct.resize(kCKeys);
    for (int k = 0; k < kWKeys; k++) h->wt[k] = (uint16_t)std::rint(32768.0 * std::exp(-centre_distance(k, kWMant)));
    for (int k = 0; k < kCKeys; k++) h->ct[k] = (uint16_t)std::rint(4096.0 * centre_distance(k, kCMant));

    auto pack = [&](int n, const std::vector<int16_t> &pal, std::vector<int32_t> &pk, std::vector<uint32_t> &n2) {
        pk.assign((size_t)n * F, 0);
        n2.assign(n, 0);
        for (int a = 0; a < n; a++) {
            uint32_t s = 0;
            for (int k = 0; k < F; k++) {
                const int16_t lo = pal[(size_t)a * twoF + 2 * k], hi = pal[(size_t)a * twoF + 2 * k + 1];
                pk[(size_t)a * F + k] = (int32_t)(((uint32_t)(uint16_t)lo) | ((uint32_t)(uint16_t)hi << 16));
                s += (uint32_t)(lo * lo) + (uint32_t)(hi * hi);
            }
            n2[a] = s;
        }
    };
    std::vector<int32_t> pkx, pky;
    std::vector<uint32_t> n2x, n2y;
    pack(bins_w, h->pal_x, pkx, n2x);
    pack(bins_h, h->pal_y, pky, n2y);

    // one allocation: constants, replicated histograms, last histogram, peak list, counters
    size_t off = 0;
    auto carve = [&](size_t bytes) {
        const size_t o = off;
        off = align_up(off + bytes, 256);
        return o;
    };
    const size_t o_px = carve(pkx.size() * 4), o_py = carve(pky.size() * 4);
    const size_t o_nx = carve(n2x.size() * 4), o_ny = carve(n2y.size() * 4);
    const size_t o_wt = carve(kWKeys * 2), o_ct = carve(kCKeys * 2);
    const size_t o_cx = carve(cx.size() * 4), o_cy = carve(cy.size() * 4);
    const size_t o_hrep = carve((size_t)kReplicas * nb * 8);
    const size_t o_hlast = carve((size_t)nb * 8);
    const size_t o_peaks = carve((size_t)centroid_capacity * 4);
    const size_t o_kinfo = carve(16);
    h->dev_bytes = off;
    if (hipMalloc(&h->dev, off) != hipSuccess) {
        delete h;
        return CPE_ERR_OUT_OF_MEMORY;
    }
    unsigned char *d = h->dev;
    bool ok = hipMemcpy(d + o_px, pkx.data(), pkx.size() * 4, hipMemcpyHostToDevice) == hipSuccess &&
              hipMemcpy(d + o_py, pky.data(), pky.size() * 4, hipMemcpyHostToDevice) == hipSuccess &&
              hipMemcpy(d + o_nx, n2x.data(), n2x.size() * 4, hipMemcpyHostToDevice) == hipSuccess &&
              hipMemcpy(d + o_ny, n2y.data(), n2y.size() * 4, hipMemcpyHostToDevice) == hipSuccess &&
              hipMemcpy(d + o_wt, h->wt.data(), kWKeys * 2, hipMemcpyHostToDevice) == hipSuccess &&
              hipMemcpy(d + o_ct, h->ct.data(), kCKeys * 2, hipMemcpyHostToDevice) == hipSuccess &&
              hipMemcpy(d + o_cx, cx.data(), cx.size() * 4, hipMemcpyHostToDevice) == hipSuccess &&
              hipMemcpy(d + o_cy, cy.data(), cy.size() * 4, hipMemcpyHostToDevice) == hipSuccess &&
              hipMemset(d + o_hrep, 0, (size_t)kReplicas * nb * 8) == hipSuccess &&
              hipMemset(d + o_hlast, 0, (size_t)nb * 8) == hipSuccess &&
              hipMemset(d + o_kinfo, 0, 16) == hipSuccess && hipDeviceSynchronize() == hipSuccess;
    if (!ok) {
        (void)hipFree(h->dev);
        delete h;
        return CPE_ERR_HIP;
    }
    h->tb.pal_x = reinterpret_cast<const int32_t *>(d + o_px);
    h->tb.pal_y = reinterpret_cast<const int32_t *>(d + o_py);
    h->tb.n2_x = reinterpret_cast<const uint32_t *>(d + o_nx);
    h->tb.n2_y = reinterpret_cast<const uint32_t *>(d + o_ny);
    h->tb.wt = reinterpret_cast<const uint16_t *>(d + o_wt);
    h->tb.ct = reinterpret_cast<const uint16_t *>(d + o_ct);
    h->tb.cx = reinterpret_cast<const float *>(d + o_cx);
    h->tb.cy = reinterpret_cast<const float *>(d + o_cy);
    h->hrep = reinterpret_cast<unsigned long long *>(d + o_hrep);
    h->hlast = reinterpret_cast<unsigned long long *>(d + o_hlast);
    h->peaks = reinterpret_cast<int32_t *>(d + o_peaks);
    h->kinfo = reinterpret_cast<int32_t *>(d + o_kinfo);
    *out = h;
    return CPE_OK;
}

cpe_status cpe_decode(cpe_decoder *h, hipStream_t stream, const void *emb, const void *fg, int32_t H, int32_t W,
                      float fg_threshold, double peak_threshold, cpe_centroid *centroids, int32_t *num_centroids,
                      int32_t *labels, float *score_map)
{
    if (!h || !emb || !fg || !centroids || !num_centroids || !labels) return CPE_ERR_INVALID_ARG;
    if (H != h->H || W != h->W) return CPE_ERR_INVALID_ARG;
    const size_t esz = h->dtype == CPE_F32 ? 4 : 2;
    if (!aligned(emb, 16) || !aligned(fg, esz) || !aligned(labels, 16) || !aligned(centroids, 8) ||
        !aligned(num_centroids, 4) || (score_map && !aligned(score_map, 4)))
        return CPE_ERR_INVALID_ARG;
    if (!std::isfinite(fg_threshold) || !std::isfinite(peak_threshold)) return CPE_ERR_INVALID_ARG;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return CPE_ERR_HIP;
    if (dev != h->device) return CPE_ERR_INVALID_ARG;
    const long long cut = peak_cut(peak_threshold);
    if (h->dtype == CPE_F32)
        return dispatch_f<float>(h, stream, emb, fg, fg_threshold, cut, centroids, num_centroids, labels, score_map);
    return dispatch_f<_Float16>(h, stream, emb, fg, fg_threshold, cut, centroids, num_centroids, labels, score_map);
}

cpe_status cpe_decode_destroy(cpe_decoder *h)
{
    if (!h) return CPE_OK;
    const hipError_t e = hipFree(h->dev);
    delete h;
    return e == hipSuccess ? CPE_OK : CPE_ERR_HIP;
}

cpe_status cpe_decode_get_tables(const cpe_decoder *h, int16_t *pal_x, int16_t *pal_y, uint16_t *weights,
                                 uint16_t *codes)
{
    if (!h) return CPE_ERR_INVALID_ARG;
    if (pal_x) std::memcpy(pal_x, h->pal_x.data(), h->pal_x.size() * sizeof(int16_t));
    if (pal_y) std::memcpy(pal_y, h->pal_y.data(), h->pal_y.size() * sizeof(int16_t));
    if (weights) std::memcpy(weights, h->wt.data(), h->wt.size() * sizeof(uint16_t));
    if (codes) std::memcpy(codes, h->ct.data(), h->ct.size() * sizeof(uint16_t));
    return CPE_OK;
}

cpe_status cpe_decode_get_histogram(cpe_decoder *h, hipStream_t stream, uint64_t *hist)
{
    if (!h || !hist || !aligned(hist, 8)) return CPE_ERR_INVALID_ARG;
    const size_t bytes = (size_t)h->bins_w * h->bins_h * 8;
    return hipMemcpyAsync(hist, h->hlast, bytes, hipMemcpyDeviceToDevice, stream) == hipSuccess ? CPE_OK : CPE_ERR_HIP;
}

size_t cpe_decode_workspace_bytes(const cpe_decoder *h) { return h ? h->dev_bytes : 0; }

cpe_status cpe_decode_set_stage_events(cpe_decoder *h, hipEvent_t *events, int32_t n_events)
{
    if (!h) return CPE_ERR_INVALID_ARG;
    if (!events) {
        h->stage_on = false;
        return CPE_OK;
    }
    if (n_events != CPE_STAGE_EVENTS) return CPE_ERR_INVALID_ARG;
    for (int i = 0; i < CPE_STAGE_EVENTS; i++) {
        if (!events[i]) return CPE_ERR_INVALID_ARG;
        h->stage_ev[i] = events[i];
    }
    h->stage_on = true;
    return CPE_OK;
}

}  // extern "C"
