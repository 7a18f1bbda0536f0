// gfx950 kernels of libsame: table build, colour-group Gibbs sweep, count
// histogram, moving sum, Gamma/Dirichlet resample.
//
// Data layout (HBM): states [n][m][ld] int8 (or int16), obs [n][ld] uint8.
// A lane owns 4 consecutive columns of one (node, replica): one dword of int8
// states (8 bytes for int16), one dword of obs bytes, and exactly one Philox
// block (4 words = the 4 columns' uniforms).  Consecutive lanes own
// consecutive column quads, so every state and obs load of a wavefront is a
// contiguous 256-byte (int8) segment.
#include <hip/hip_runtime.h>

#include <cfloat>
#include <cstdint>

#include "launch.hpp"
#include "philox.hpp"

namespace same {
namespace dev {

constexpr int kBlock = 256;          // 4 wavefronts of 64
constexpr int kColsPerBlock = 4 * kBlock;
constexpr int kHistBins = 4096;      // LDS histogram capacity (16 KB)
constexpr float kUnderflowGuard = 0x1p-100f;

// ---------------------------------------------------------------- state quads

template <typename ST>
struct Quad;

template <>
struct Quad<int8_t> {
    using V = uint32_t;
    __device__ static V load(const int8_t *p) { return *reinterpret_cast<const uint32_t *>(p); }
    __device__ static void store(int8_t *p, V v) { *reinterpret_cast<uint32_t *>(p) = v; }
    __device__ static int get(V v, int c) { return (int)((v >> (8 * c)) & 0xffu); }
    __device__ static V put(V v, int c, int x) {
        return (v & ~(0xffu << (8 * c))) | ((uint32_t)x << (8 * c));
    }
    // keeps the first nvalid (1..4) columns, zeroes the rest
    __device__ static V keep(V v, int nvalid) {
        return nvalid >= 4 ? v : (v & ((1u << (8 * nvalid)) - 1u));
    }
};

template <>
struct Quad<int16_t> {
    using V = uint2;
    __device__ static V load(const int16_t *p) { return *reinterpret_cast<const uint2 *>(p); }
    __device__ static void store(int16_t *p, V v) { *reinterpret_cast<uint2 *>(p) = v; }
    __device__ static int get(V v, int c) {
        const uint32_t w = c < 2 ? v.x : v.y;
        return (int)((w >> (16 * (c & 1))) & 0xffffu);
    }
    __device__ static V put(V v, int c, int x) {
        const uint32_t sh = 16 * (c & 1);
        if (c < 2) v.x = (v.x & ~(0xffffu << sh)) | ((uint32_t)x << sh);
        else v.y = (v.y & ~(0xffffu << sh)) | ((uint32_t)x << sh);
        return v;
    }
    __device__ static V keep(V v, int nvalid) {
        if (nvalid >= 4) return v;
        if (nvalid <= 2) {
            v.y = 0;
            if (nvalid == 1) v.x &= 0xffffu;
        } else {
            v.y &= 0xffffu;
        }
        return v;
    }
};

// Reads one k-vector of KP floats (KP <= KPMAX, both powers of two) into f;
// entries KP..KPMAX-1 become zero.  p is 8-byte aligned for KP == 2 and
// 16-byte aligned otherwise.
template <int KPMAX>
__device__ __forceinline__ void load_kvec(const float *__restrict__ p, int KP, float (&f)[KPMAX]) {
    if (KPMAX == 2 || KP == 2) {
        const float2 v = *reinterpret_cast<const float2 *>(p);
        f[0] = v.x;
        f[1] = v.y;
#pragma unroll
        for (int k = 2; k < KPMAX; ++k) f[k] = 0.f;
        return;
    }
#pragma unroll
    for (int q = 0; q < KPMAX / 4; ++q) {
        if (4 * q < KP) {
            const float4 v = reinterpret_cast<const float4 *>(p)[q];
            f[4 * q + 0] = v.x;
            f[4 * q + 1] = v.y;
            f[4 * q + 2] = v.z;
            f[4 * q + 3] = v.w;
        } else {
            f[4 * q + 0] = f[4 * q + 1] = f[4 * q + 2] = f[4 * q + 3] = 0.f;
        }
    }
}

// Exact power-of-two rescale so that max_k w[k] lands in [0.5, 1).
template <int KPMAX>
__device__ __forceinline__ void renorm(float (&w)[KPMAX]) {
    float mx = w[0];
#pragma unroll
    for (int k = 1; k < KPMAX; ++k) mx = fmaxf(mx, w[k]);
    if (mx > 0.f) {
        const int e = __builtin_amdgcn_frexp_expf(mx);
#pragma unroll
        for (int k = 0; k < KPMAX; ++k) w[k] = __builtin_ldexpf(w[k], -e);
    }
}

// Unnormalised full conditional of the block's node for the lane's 4 columns:
// w[c][k] = own k-vector * product over children of the child k-vectors.
// With RESCALE the running product of each column is renormalised after every
// factor, which keeps it away from fp32 underflow at the cost of ~2*KP extra
// ops per factor; the default path checks the final maximum instead.
// Columns at or beyond n_cols (only in the last quad; nvalid < 4) read their
// states as 0, so padding never steers a table index out of range.
template <int KPMAX, typename ST, bool RESCALE>
__device__ __forceinline__ void blanket_product(const int32_t *__restrict__ d,
                                                const float *__restrict__ table,
                                                const ST *__restrict__ base, int64_t vstride,
                                                int nvalid, float (&w)[4][KPMAX]) {
    using Q = Quad<ST>;
    const int KP = d[1];
    const int n_par = d[3];
    const int n_child = d[4];
    const int32_t *p = d + 5;
    int a[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) a[c] = d[2];
    for (int q = 0; q < n_par; ++q, p += 2) {
        const typename Q::V s = Q::keep(Q::load(base + (int64_t)p[0] * vstride), nvalid);
        const int mult = p[1];
#pragma unroll
        for (int c = 0; c < 4; ++c) a[c] += Q::get(s, c) * mult;
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) load_kvec<KPMAX>(table + a[c], KP, w[c]);
    for (int h = 0; h < n_child; ++h) {
        const int hn = p[0], toff = p[1], xmul = p[2], ncop = p[3];
        p += 4;
        const typename Q::V xs = Q::keep(Q::load(base + (int64_t)hn * vstride), nvalid);
        int b[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) b[c] = toff + Q::get(xs, c) * xmul;
        for (int q = 0; q < ncop; ++q, p += 2) {
            const typename Q::V s = Q::keep(Q::load(base + (int64_t)p[0] * vstride), nvalid);
            const int mult = p[1];
#pragma unroll
            for (int c = 0; c < 4; ++c) b[c] += Q::get(s, c) * mult;
        }
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            float f[KPMAX];
            load_kvec<KPMAX>(table + b[c], KP, f);
#pragma unroll
            for (int k = 0; k < KPMAX; ++k) w[c][k] *= f[k];
            if (RESCALE) renorm<KPMAX>(w[c]);
        }
    }
}

// Inverse-CDF draw from weights w[0..K) (entries K..KPMAX-1 are zero):
// S_k running sums in ascending k, Z = S_{K-1}; the smallest k with u*Z < S_k,
// else the largest k with positive weight.
template <int KPMAX>
__device__ __forceinline__ int draw_kvec(float (&w)[KPMAX], int K, float u, float &Z) {
    float S[KPMAX];
    float acc = 0.f;
#pragma unroll
    for (int k = 0; k < KPMAX; ++k) {
        acc += w[k];
        S[k] = acc;
    }
    Z = acc;
    const float t = u * Z;
    int pick = 0;
#pragma unroll
    for (int k = 0; k < KPMAX; ++k) pick += (S[k] <= t) ? 1 : 0;
    if (pick >= K) {
        pick = 0;
#pragma unroll
        for (int k = 0; k < KPMAX; ++k)
            if (k < K && w[k] > 0.f) pick = k;
    }
    return pick;
}

template <int KPMAX, typename ST, bool DEBUG>
__global__ __launch_bounds__(kBlock) void sweep_color_kernel(
    const int32_t *__restrict__ desc, const int32_t *__restrict__ desc_off,
    const int32_t *__restrict__ order, int32_t begin, const float *__restrict__ table,
    ST *__restrict__ states, const uint8_t *__restrict__ obs, int32_t m, int64_t n_cols, int64_t ld,
    int64_t col_offset, uint32_t key0, uint32_t key1, uint32_t sweep_id, int64_t win_begin,
    int64_t win, float *__restrict__ probs, int32_t max_card) {
    using Q = Quad<ST>;
    const int node = order[begin + blockIdx.z];
    const int r = blockIdx.y;
    const int64_t col = ((int64_t)blockIdx.x * kBlock + threadIdx.x) * 4;
    if (col >= n_cols) return;
    const int32_t *__restrict__ d = desc + desc_off[node];
    const int K = d[0];

    const uint32_t ob = *reinterpret_cast<const uint32_t *>(obs + (int64_t)node * ld + col);
    bool lat[4];
    bool any = false;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        lat[c] = ((ob >> (8 * c)) & 0xffu) == 0 && col + c < n_cols;
        any |= lat[c];
    }
    if (!any) return;

    const int64_t vstride = (int64_t)m * ld;
    const ST *base = states + (int64_t)r * ld + col;
    const int nvalid = n_cols - col < 4 ? (int)(n_cols - col) : 4;
    float w[4][KPMAX];
    blanket_product<KPMAX, ST, false>(d, table, base, vstride, nvalid, w);
    bool low = false;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        float mx = w[c][0];
#pragma unroll
        for (int k = 1; k < KPMAX; ++k) mx = fmaxf(mx, w[c][k]);
        low |= lat[c] && !(mx >= kUnderflowGuard);
    }
    if (low) blanket_product<KPMAX, ST, true>(d, table, base, vstride, nvalid, w);

    const uint64_t g = (uint64_t)(col_offset + col);
    const Philox4 rnd = philox4x32_10((uint32_t)(g >> 2), (uint32_t)node, (uint32_t)r, sweep_id,
                                      key0, key1);
    ST *own = states + ((int64_t)node * m + r) * ld + col;
    typename Q::V cur = Q::load(own);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        if (!lat[c]) continue;
        const float u = (float)(rnd.w[c] >> 8) * 0x1p-24f;
        float Z;
        const int x = draw_kvec<KPMAX>(w[c], K, u, Z);
        cur = Q::put(cur, c, x);
        if (DEBUG) {
            const int64_t j = col + c;
            if (j >= win_begin && j < win_begin + win) {
                float *dst = probs + (((int64_t)node * m + r) * win + (j - win_begin)) * max_card;
                for (int k = 0; k < K; ++k) dst[k] = w[c][k] / Z;
            }
        }
    }
    Q::store(own, cur);
}

// ------------------------------------------------- generic path, K_i > 16
//
// The weight of state k is kept as (mantissa in [0.5, 1), exponent) and
// renormalised exactly after every factor, so any K fits in a few registers;
// the three passes (largest exponent, total, search) each recompute the
// products.

template <typename ST>
__device__ float weight_ext(const int32_t *__restrict__ d, const float *__restrict__ table,
                            const ST *__restrict__ base, int64_t vstride, int c, int k, int &e) {
    using Q = Quad<ST>;
    const int n_par = d[3];
    const int n_child = d[4];
    const int32_t *p = d + 5;
    int a = d[2];
    for (int q = 0; q < n_par; ++q, p += 2)
        a += Q::get(Q::load(base + (int64_t)p[0] * vstride), c) * p[1];
    float mnt = table[a + k];
    e = 0;
    for (int h = 0; h < n_child; ++h) {
        const int hn = p[0], toff = p[1], xmul = p[2], ncop = p[3];
        p += 4;
        int b = toff + Q::get(Q::load(base + (int64_t)hn * vstride), c) * xmul;
        for (int q = 0; q < ncop; ++q, p += 2)
            b += Q::get(Q::load(base + (int64_t)p[0] * vstride), c) * p[1];
        mnt *= table[b + k];
        const int de = __builtin_amdgcn_frexp_expf(mnt);
        mnt = __builtin_ldexpf(mnt, -de);
        e += de;
    }
    return mnt;
}

template <typename ST, bool DEBUG>
__global__ __launch_bounds__(kBlock) void sweep_color_generic_kernel(
    const int32_t *__restrict__ desc, const int32_t *__restrict__ desc_off,
    const int32_t *__restrict__ order, int32_t begin, const float *__restrict__ table,
    ST *__restrict__ states, const uint8_t *__restrict__ obs, int32_t m, int64_t n_cols, int64_t ld,
    int64_t col_offset, uint32_t key0, uint32_t key1, uint32_t sweep_id, int64_t win_begin,
    int64_t win, float *__restrict__ probs, int32_t max_card) {
    using Q = Quad<ST>;
    const int node = order[begin + blockIdx.z];
    const int r = blockIdx.y;
    const int64_t col = ((int64_t)blockIdx.x * kBlock + threadIdx.x) * 4;
    if (col >= n_cols) return;
    const int32_t *__restrict__ d = desc + desc_off[node];
    const int K = d[0];
    const uint32_t ob = *reinterpret_cast<const uint32_t *>(obs + (int64_t)node * ld + col);
    const int64_t vstride = (int64_t)m * ld;
    const ST *base = states + (int64_t)r * ld + col;
    const uint64_t g = (uint64_t)(col_offset + col);
    const Philox4 rnd = philox4x32_10((uint32_t)(g >> 2), (uint32_t)node, (uint32_t)r, sweep_id,
                                      key0, key1);
    ST *own = states + ((int64_t)node * m + r) * ld + col;
    typename Q::V cur = Q::load(own);
    for (int c = 0; c < 4; ++c) {
        if (((ob >> (8 * c)) & 0xffu) != 0 || col + c >= n_cols) continue;
        int E = -100000;
        for (int k = 0; k < K; ++k) {
            int e;
            const float mk = weight_ext<ST>(d, table, base, vstride, c, k, e);
            if (mk > 0.f && e > E) E = e;
        }
        float Z = 0.f;
        for (int k = 0; k < K; ++k) {
            int e;
            const float mk = weight_ext<ST>(d, table, base, vstride, c, k, e);
            Z += __builtin_ldexpf(mk, e - E);
        }
        const float t = (float)(rnd.w[c] >> 8) * 0x1p-24f * Z;
        float S = 0.f;
        int pick = -1, last_pos = 0;
        for (int k = 0; k < K; ++k) {
            int e;
            const float wk = __builtin_ldexpf(weight_ext<ST>(d, table, base, vstride, c, k, e), e - E);
            S += wk;
            if (wk > 0.f) last_pos = k;
            if (pick < 0 && t < S) pick = k;
            if (DEBUG) {
                const int64_t j = col + c;
                if (j >= win_begin && j < win_begin + win)
                    probs[(((int64_t)node * m + r) * win + (j - win_begin)) * max_card + k] = wk / Z;
            }
        }
        if (pick < 0) pick = last_pos;
        cur = Q::put(cur, c, pick);
    }
    Q::store(own, cur);
}

// ---------------------------------------------------------------- table build

__global__ __launch_bounds__(kBlock) void build_tables_kernel(
    const Segment *__restrict__ segs, const int32_t *__restrict__ blk_seg,
    const int32_t *__restrict__ blk_first, const float *__restrict__ cpts, float *__restrict__ table) {
    const Segment sg = segs[blk_seg[blockIdx.x]];
    const int32_t grp = blk_first[blockIdx.x] + (int32_t)threadIdx.x;
    if (grp >= sg.n_groups) return;
    int64_t src, step;
    if (sg.own) {
        src = sg.src + (int64_t)grp * sg.K;
        step = 1;
    } else {
        const int64_t up = grp / sg.Kh, xh = grp % sg.Kh;
        const int64_t ufull = (up / sg.s) * sg.s * sg.K + (up % sg.s);
        src = sg.src + ufull * sg.Kh + xh;
        step = (int64_t)sg.s * sg.Kh;
    }
    float mx = FLT_MIN;
    for (int k = 0; k < sg.K; ++k) mx = fmaxf(mx, cpts[src + k * step]);
    const int e = __builtin_amdgcn_frexp_expf(mx);
    float *dst = table + sg.dst + (int64_t)grp * sg.KP;
    for (int k = 0; k < sg.K; ++k)
        dst[k] = __builtin_ldexpf(fmaxf(cpts[src + k * step], FLT_MIN), -e);
    for (int k = sg.K; k < sg.KP; ++k) dst[k] = 0.f;
}

// ---------------------------------------------------------------- counts

__global__ void fill_zero_kernel(int32_t *p, int64_t count) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

template <typename ST>
__global__ __launch_bounds__(kBlock) void count_kernel(const int32_t *__restrict__ cdesc,
                                                      const int32_t *__restrict__ cdesc_off,
                                                      int32_t node_base,
                                                      const ST *__restrict__ states, int32_t m,
                                                      int64_t n_cols, int64_t ld,
                                                      int32_t *__restrict__ counts) {
    using Q = Quad<ST>;
    __shared__ int32_t hist[kHistBins];
    const int node = node_base + (int)blockIdx.z;
    const int r = blockIdx.y;
    const int32_t *__restrict__ d = cdesc + cdesc_off[node];
    const int K = d[0], n_par = d[1], nbins = d[2], off = d[3];
    const bool use_lds = nbins <= kHistBins;
    if (use_lds)
        for (int b = threadIdx.x; b < nbins; b += kBlock) hist[b] = 0;
    __syncthreads();
    const int64_t col = ((int64_t)blockIdx.x * kBlock + threadIdx.x) * 4;
    if (col < n_cols) {
        const int64_t vstride = (int64_t)m * ld;
        const ST *base = states + (int64_t)r * ld + col;
        int u[4] = {0, 0, 0, 0};
        const int32_t *p = d + 4;
        for (int q = 0; q < n_par; ++q, p += 2) {
            const typename Q::V s = Q::load(base + (int64_t)p[0] * vstride);
#pragma unroll
            for (int c = 0; c < 4; ++c) u[c] += Q::get(s, c) * p[1];
        }
        const typename Q::V xs = Q::load(base + (int64_t)node * vstride);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            if (col + c >= n_cols) break;
            const int bin = u[c] * K + Q::get(xs, c);
            if (use_lds) atomicAdd(&hist[bin], 1);
            else atomicAdd(&counts[off + bin], 1);
        }
    }
    if (use_lds) {
        __syncthreads();
        for (int b = threadIdx.x; b < nbins; b += kBlock) {
            const int v = hist[b];
            if (v) atomicAdd(&counts[off + b], v);
        }
    }
}

__global__ void moving_sum_kernel(const int32_t *__restrict__ newc, int32_t *__restrict__ mb,
                                  int32_t *__restrict__ totals, int64_t total) {
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int32_t nv = newc[e];
        const int32_t delta = nv - mb[e];
        mb[e] = nv;
        if (totals) totals[e] += delta;
    }
}

// ---------------------------------------------------------------- Dirichlet

// Gamma(a, 1), Marsaglia & Tsang (2000), fp64, with the a < 1 boost
// Gamma(a) = Gamma(a + 1) * U^(1/a).  Attempt t uses the Philox block at
// counter {e, t, 1 << 24, q}: Box-Muller normal from words 0 and 1, the
// acceptance uniform from word 2 and the boost uniform from word 3.
__device__ double gamma_mt(double a, uint32_t e, uint32_t q, uint32_t k0, uint32_t k1) {
#pragma clang fp contract(off)
    const bool boost = a < 1.0;
    const double b = boost ? a + 1.0 : a;
    const double d = b - 1.0 / 3.0;
    const double c = 1.0 / sqrt(9.0 * d);
    for (uint32_t t = 0; t < 256; ++t) {
        const Philox4 w = philox4x32_10(e, t, 1u << 24, q, k0, k1);
        const double u1 = ((double)(w.w[0] >> 8) + 1.0) * 0x1p-24;
        const double u2 = (double)(w.w[1] >> 8) * 0x1p-24;
        const double z = sqrt(-2.0 * log(u1)) * cos(6.283185307179586476925286766559 * u2);
        double v = 1.0 + c * z;
        if (v <= 0.0) continue;
        v = v * v * v;
        const double ua = ((double)(w.w[2] >> 8) + 1.0) * 0x1p-24;
        if (log(ua) < 0.5 * z * z + d - d * v + d * log(v)) {
            double gv = d * v;
            if (boost) gv *= pow(((double)(w.w[3] >> 8) + 1.0) * 0x1p-24, 1.0 / a);
            return gv;
        }
    }
    return d;
}

__global__ void gamma_kernel(const int32_t *__restrict__ totals, double alpha, uint32_t k0,
                             uint32_t k1, uint32_t update_id, double *__restrict__ g, int64_t total) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= total) return;
    g[e] = gamma_mt(alpha + (double)totals[e], (uint32_t)e, update_id, k0, k1);
}

__global__ void normalize_kernel(const int32_t *__restrict__ row_off, const int32_t *__restrict__ row_k,
                                 const double *__restrict__ g, float *__restrict__ cpts,
                                 int64_t n_rows) {
#pragma clang fp contract(off)
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= n_rows) return;
    const int64_t o = row_off[r];
    const int K = row_k[r];
    double s = 0.0;
    for (int k = 0; k < K; ++k) s += g[o + k];
    for (int k = 0; k < K; ++k) cpts[o + k] = (float)(s > 0.0 ? g[o + k] / s : 1.0 / K);
}

}  // namespace dev

// ================================================================= launchers

namespace {
inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }
}  // namespace

hipError_t launch_build_tables(const DeviceTables &t, const float *cpts, float *table,
                               hipStream_t stream) {
    if (t.n_build_blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(dev::build_tables_kernel, dim3(t.n_build_blocks), dim3(dev::kBlock), 0,
                       stream, t.segs, t.blk_seg, t.blk_first, cpts, table);
    return hipGetLastError();
}

namespace {

template <int KPMAX, typename ST>
void sweep_variant(const SweepArgs &a, int32_t begin, int32_t count, dim3 grid, hipStream_t stream) {
    grid.z = count;
    if (a.win > 0)
        hipLaunchKernelGGL((dev::sweep_color_kernel<KPMAX, ST, true>), grid, dim3(dev::kBlock), 0,
                           stream, a.t->desc, a.t->desc_off, a.t->order, begin, a.table,
                           (ST *)a.states, a.obs, a.m, a.n_cols, a.ld, a.col_offset, a.key0, a.key1,
                           a.sweep_id, a.win_begin, a.win, a.probs, a.max_card);
    else
        hipLaunchKernelGGL((dev::sweep_color_kernel<KPMAX, ST, false>), grid, dim3(dev::kBlock), 0,
                           stream, a.t->desc, a.t->desc_off, a.t->order, begin, a.table,
                           (ST *)a.states, a.obs, a.m, a.n_cols, a.ld, a.col_offset, a.key0, a.key1,
                           a.sweep_id, a.win_begin, a.win, a.probs, a.max_card);
}

template <typename ST>
void sweep_generic(const SweepArgs &a, int32_t begin, int32_t count, dim3 grid, hipStream_t stream) {
    grid.z = count;
    if (a.win > 0)
        hipLaunchKernelGGL((dev::sweep_color_generic_kernel<ST, true>), grid, dim3(dev::kBlock), 0,
                           stream, a.t->desc, a.t->desc_off, a.t->order, begin, a.table,
                           (ST *)a.states, a.obs, a.m, a.n_cols, a.ld, a.col_offset, a.key0, a.key1,
                           a.sweep_id, a.win_begin, a.win, a.probs, a.max_card);
    else
        hipLaunchKernelGGL((dev::sweep_color_generic_kernel<ST, false>), grid, dim3(dev::kBlock), 0,
                           stream, a.t->desc, a.t->desc_off, a.t->order, begin, a.table,
                           (ST *)a.states, a.obs, a.m, a.n_cols, a.ld, a.col_offset, a.key0, a.key1,
                           a.sweep_id, a.win_begin, a.win, a.probs, a.max_card);
}

template <typename ST>
void sweep_dispatch(const SweepArgs &a, int32_t begin, int32_t count, int32_t kp, dim3 grid,
                    hipStream_t stream) {
    switch (kp) {
        case 2: sweep_variant<2, ST>(a, begin, count, grid, stream); break;
        case 4: sweep_variant<4, ST>(a, begin, count, grid, stream); break;
        case 8: sweep_variant<8, ST>(a, begin, count, grid, stream); break;
        case 16: sweep_variant<16, ST>(a, begin, count, grid, stream); break;
        default: sweep_generic<ST>(a, begin, count, grid, stream); break;
    }
}

}  // namespace

hipError_t launch_sweep_color(const SweepArgs &a, int32_t begin, int32_t count, int32_t kp,
                              int32_t state_bytes, hipStream_t stream) {
    if (count <= 0 || a.n_cols <= 0) return hipSuccess;
    dim3 grid(blocks_for(a.n_cols, dev::kColsPerBlock), (unsigned)a.m, 1);
    for (int32_t s = 0; s < count; s += 65535) {
        const int32_t c = count - s < 65535 ? count - s : 65535;
        if (state_bytes == 1) sweep_dispatch<int8_t>(a, begin + s, c, kp, grid, stream);
        else sweep_dispatch<int16_t>(a, begin + s, c, kp, grid, stream);
    }
    return hipGetLastError();
}

hipError_t launch_fill_zero(int32_t *p, int64_t count, hipStream_t stream) {
    if (count <= 0) return hipSuccess;
    unsigned nb = blocks_for(count, dev::kBlock);
    if (nb > 4096) nb = 4096;
    hipLaunchKernelGGL(dev::fill_zero_kernel, dim3(nb), dim3(dev::kBlock), 0, stream, p, count);
    return hipGetLastError();
}

hipError_t launch_counts(const DeviceTables &t, const void *states, int32_t state_bytes,
                         int32_t n, int32_t m, int64_t n_cols, int64_t ld, int32_t *counts,
                         hipStream_t stream) {
    if (n_cols <= 0) return hipSuccess;
    for (int32_t s = 0; s < n; s += 65535) {
        const int32_t c = n - s < 65535 ? n - s : 65535;
        dim3 grid(blocks_for(n_cols, dev::kColsPerBlock), (unsigned)m, (unsigned)c);
        if (state_bytes == 1)
            hipLaunchKernelGGL(dev::count_kernel<int8_t>, grid, dim3(dev::kBlock), 0, stream, t.cdesc,
                               t.cdesc_off, s, (const int8_t *)states, m, n_cols, ld, counts);
        else
            hipLaunchKernelGGL(dev::count_kernel<int16_t>, grid, dim3(dev::kBlock), 0, stream, t.cdesc,
                               t.cdesc_off, s, (const int16_t *)states, m, n_cols, ld, counts);
    }
    return hipGetLastError();
}

hipError_t launch_moving_sum(const int32_t *newc, int32_t *mb, int32_t *totals, int64_t total,
                             hipStream_t stream) {
    if (total <= 0) return hipSuccess;
    unsigned nb = blocks_for(total, dev::kBlock);
    if (nb > 4096) nb = 4096;
    hipLaunchKernelGGL(dev::moving_sum_kernel, dim3(nb), dim3(dev::kBlock), 0, stream, newc, mb,
                       totals, total);
    return hipGetLastError();
}

hipError_t launch_gamma(const int32_t *totals, double alpha, uint32_t key0, uint32_t key1,
                        uint32_t update_id, double *g, int64_t total, hipStream_t stream) {
    if (total <= 0) return hipSuccess;
    hipLaunchKernelGGL(dev::gamma_kernel, dim3(blocks_for(total, dev::kBlock)), dim3(dev::kBlock), 0,
                       stream, totals, alpha, key0, key1, update_id, g, total);
    return hipGetLastError();
}

hipError_t launch_normalize(const DeviceTables &t, const double *g, float *cpts, int64_t n_rows,
                            hipStream_t stream) {
    if (n_rows <= 0) return hipSuccess;
    hipLaunchKernelGGL(dev::normalize_kernel, dim3(blocks_for(n_rows, dev::kBlock)), dim3(dev::kBlock),
                       0, stream, t.row_off, t.row_k, g, cpts, n_rows);
    return hipGetLastError();
}

}  // namespace same
