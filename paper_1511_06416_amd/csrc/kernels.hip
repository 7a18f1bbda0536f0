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

// Structure tables are read through the constant address space: their
// addresses are uniform across a block, so the reads become scalar loads
// served by the scalar cache instead of vector memory round trips.
typedef const __attribute__((address_space(4))) int32_t cint32_t;

__device__ __forceinline__ cint32_t *as_const(const int32_t *p) { return (cint32_t *)p; }

constexpr int kBlock = 256;          // 4 wavefronts of 64
constexpr int kColsPerBlock = 4 * kBlock;
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

// Reads one k-vector of KP floats (KP a power of two); p is 8-byte aligned
// for KP == 2 and 16-byte aligned otherwise.
template <int KP>
__device__ __forceinline__ void load_kvec(const float *__restrict__ p, float (&f)[KP]) {
    if (KP == 2) {
        const float2 v = *reinterpret_cast<const float2 *>(p);
        f[0] = v.x;
        f[1] = v.y;
        return;
    }
#pragma unroll
    for (int q = 0; q < KP / 4; ++q) {
        const float4 v = reinterpret_cast<const float4 *>(p)[q];
        f[4 * q + 0] = v.x;
        f[4 * q + 1] = v.y;
        f[4 * q + 2] = v.z;
        f[4 * q + 3] = v.w;
    }
}

// Exact power-of-two rescale so that max_k w[k] lands in [0.5, 1).
template <int KP>
__device__ __forceinline__ void renorm(float (&w)[KP]) {
    float mx = w[0];
#pragma unroll
    for (int k = 1; k < KP; ++k) mx = fmaxf(mx, w[k]);
    if (mx > 0.f) {
        const int e = __builtin_amdgcn_frexp_expf(mx);
#pragma unroll
        for (int k = 0; k < KP; ++k) w[k] = __builtin_ldexpf(w[k], -e);
    }
}

constexpr int kEntryBatch = 8;  // state rows loaded per batch (one round trip)

// Loads the state quads of up to kEntryBatch entries starting at e0.  Every
// slot loads (slots past the end reload entry e0), so the whole batch is in
// flight before the first use.
//
// Addressing: the row base states + node * m * ld is uniform (scalar), the
// lane's offset (r * ld + col) is shared by every row and fits 32 bits (the
// host requires m * ld * sizeof(state) < 2^31), so every load is a scalar
// base plus one 32-bit vector offset.
template <typename ST>
__device__ __forceinline__ void load_batch(cint32_t *ent, int e0, int ne, const ST *__restrict__ states,
                                           uint32_t lane_off, int64_t vstride,
                                           typename Quad<ST>::V (&s)[kEntryBatch]) {
#pragma unroll
    for (int t = 0; t < kEntryBatch; ++t) {
        const int tt = t < ne ? e0 + t : e0;
        const ST *row = states + (int64_t)ent[3 * tt] * vstride;
        s[t] = Quad<ST>::load(row + lane_off);
    }
}

// Multiplies the k-vectors at tab + b[c] into w[c] (renormalising with RESCALE).
template <int KP, bool RESCALE>
__device__ __forceinline__ void mul_kvecs(const float *tab, const int (&b)[4], float (&w)[4][KP]) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        float f[KP];
        load_kvec<KP>(tab + b[c], f);
#pragma unroll
        for (int k = 0; k < KP; ++k) w[c][k] *= f[k];
        if (RESCALE) renorm<KP>(w[c]);
    }
}

// Unnormalised full conditional of a node for the 4 columns of one quad from
// its product-path entry list: w[c][k] = own k-vector * product over children
// of the child k-vectors, all read from tab (the node's table record, in LDS
// or global memory).  cur receives the node's own state quad.  With RESCALE
// each column's running product is renormalised after every factor, which
// keeps it away from fp32 underflow; the default path checks the final
// maximum instead.  Columns at or beyond n_cols (nvalid < 4, last quad only)
// read their states as 0, so padding never steers a table index out of range.
template <int KP, typename ST, bool RESCALE>
__device__ __forceinline__ void product_walk(cint32_t *ent, int n_ent, const float *tab,
                                             const ST *__restrict__ states, uint32_t lane_off,
                                             int64_t vstride, int nvalid, float (&w)[4][KP],
                                             typename Quad<ST>::V &cur) {
    using Q = Quad<ST>;
    int a[4] = {0, 0, 0, 0};
    int b[4] = {0, 0, 0, 0};
    bool in_child = false;
    for (int e0 = 0; e0 < n_ent; e0 += kEntryBatch) {
        const int ne = n_ent - e0 < kEntryBatch ? n_ent - e0 : kEntryBatch;
        typename Q::V s[kEntryBatch];
        load_batch<ST>(ent, e0, ne, states, lane_off, vstride, s);
#pragma unroll
        for (int t = 0; t < kEntryBatch; ++t) {
            if (t >= ne) break;
            const int mult = ent[3 * (e0 + t) + 1], arg = ent[3 * (e0 + t) + 2];
            if (arg == -3) {
                cur = s[t];
                continue;
            }
            const typename Q::V v = Q::keep(s[t], nvalid);
            if (arg == -1) {
#pragma unroll
                for (int c = 0; c < 4; ++c) a[c] += Q::get(v, c) * mult;
            } else if (arg == -2) {
#pragma unroll
                for (int c = 0; c < 4; ++c) b[c] += Q::get(v, c) * mult;
            } else {
                if (in_child) {
                    mul_kvecs<KP, RESCALE>(tab, b, w);
                } else {
#pragma unroll
                    for (int c = 0; c < 4; ++c) load_kvec<KP>(tab + a[c], w[c]);
                }
                in_child = true;
#pragma unroll
                for (int c = 0; c < 4; ++c) b[c] = arg + Q::get(v, c) * mult;
            }
        }
    }
    if (in_child) {
        mul_kvecs<KP, RESCALE>(tab, b, w);
    } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) load_kvec<KP>(tab + a[c], w[c]);
    }
}

// Threshold-path index walk: idx[c] = sum of mult * state over the blanket;
// cur receives the node's own state quad.
template <typename ST>
__device__ __forceinline__ void table_walk(cint32_t *ent, int n_ent, const ST *__restrict__ states,
                                           uint32_t lane_off, int64_t vstride, int nvalid,
                                           int (&idx)[4], typename Quad<ST>::V &cur) {
    using Q = Quad<ST>;
    for (int e0 = 0; e0 < n_ent; e0 += kEntryBatch) {
        const int ne = n_ent - e0 < kEntryBatch ? n_ent - e0 : kEntryBatch;
        typename Q::V s[kEntryBatch];
        load_batch<ST>(ent, e0, ne, states, lane_off, vstride, s);
#pragma unroll
        for (int t = 0; t < kEntryBatch; ++t) {
            if (t >= ne) break;
            const int mult = ent[3 * (e0 + t) + 1], arg = ent[3 * (e0 + t) + 2];
            if (arg == -3) {
                cur = s[t];
                continue;
            }
            const typename Q::V v = Q::keep(s[t], nvalid);
#pragma unroll
            for (int c = 0; c < 4; ++c) idx[c] += Q::get(v, c) * mult;
        }
    }
}

// Inverse-CDF draw from weights w[0..K) (entries K..KP-1 are zero): S_k running
// sums in ascending k, Z = S_{K-1}; the smallest k with u*Z < S_k, else the
// largest k with positive weight.
template <int KP>
__device__ __forceinline__ int draw_kvec(const float (&w)[KP], int K, float u, float &Z) {
    float S[KP];
    float acc = 0.f;
#pragma unroll
    for (int k = 0; k < KP; ++k) {
        acc += w[k];
        S[k] = acc;
    }
    Z = acc;
    const float t = u * Z;
    int pick = 0;
#pragma unroll
    for (int k = 0; k < KP; ++k) pick += (S[k] <= t) ? 1 : 0;
    if (pick >= K) {
        pick = 0;
#pragma unroll
        for (int k = 0; k < KP; ++k)
            if (k < K && w[k] > 0.f) pick = k;
    }
    return pick;
}

// The block's share of the work: a run of column quads of one node and a
// range of replicas.
struct Work {
    int node;
    cint32_t *d;
    int64_t q0, q1;
    int r0, r1;
};

__device__ __forceinline__ Work block_work(const SweepParams &P) {
    Work w;
    w.node = as_const(P.order)[P.begin + blockIdx.y];
    w.d = as_const(P.desc) + as_const(P.desc_off)[w.node];
    const int64_t nquads = (P.n_cols + 3) >> 2;
    w.q0 = (int64_t)blockIdx.x * P.quads_per_block;
    w.q1 = w.q0 + P.quads_per_block < nquads ? w.q0 + P.quads_per_block : nquads;
    w.r0 = (int)blockIdx.z * P.reps_per_block;
    w.r1 = w.r0 + P.reps_per_block < P.m ? w.r0 + P.reps_per_block : P.m;
    return w;
}

// Latent mask of a quad: bit c set when column col + c < n_cols is latent.
__device__ __forceinline__ int latent_bits(const SweepParams &P, int node, int64_t col) {
    const uint32_t ob = *reinterpret_cast<const uint32_t *>(P.obs + (int64_t)node * P.ld + col);
    int bits = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c)
        if (((ob >> (8 * c)) & 0xffu) == 0 && col + c < P.n_cols) bits |= 1 << c;
    return bits;
}

__device__ __forceinline__ void write_probs(const SweepParams &P, int node, int r, int64_t j,
                                            const float *w, int K, float Z) {
    if (j >= P.win_begin && j < P.win_begin + P.win) {
        float *dst = P.probs + (((int64_t)node * P.m + r) * P.win + (j - P.win_begin)) * P.max_card;
        for (int k = 0; k < K; ++k) dst[k] = w[k] / Z;
    }
}

__device__ __forceinline__ Philox4 gibbs_block(const SweepParams &P, int node, int r, int64_t q) {
    return philox4x32_10((uint32_t)((P.col_offset >> 2) + q), (uint32_t)node, (uint32_t)r, P.sweep_id,
                         P.key0, P.key1);
}

// Product path: the conditional from the node's k-vector tables at tab.
template <int KP, typename ST, bool DEBUG>
__device__ void sweep_product(const SweepParams &P, const Work &W, const float *tab) {
    using Q = Quad<ST>;
    cint32_t *d = W.d;
    const int K = d[0], n_ent = d[10];
    cint32_t *ent = d + d[11];
    ST *states = reinterpret_cast<ST *>(P.states);
    const int64_t vstride = (int64_t)P.m * P.ld;
    for (int64_t q = W.q0 + threadIdx.x; q < W.q1; q += kBlock) {
        const int64_t col = q * 4;
        const int lat = latent_bits(P, W.node, col);
        if (!lat) continue;
        const int nvalid = P.n_cols - col < 4 ? (int)(P.n_cols - col) : 4;
        for (int r = W.r0; r < W.r1; ++r) {
            const uint32_t lane_off = (uint32_t)(r * P.ld + col);
            float w[4][KP];
            typename Q::V cur;
            product_walk<KP, ST, false>(ent, n_ent, tab, states, lane_off, vstride, nvalid, w, cur);
            bool low = false;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                float mx = w[c][0];
#pragma unroll
                for (int k = 1; k < KP; ++k) mx = fmaxf(mx, w[c][k]);
                low |= ((lat >> c) & 1) && !(mx >= kUnderflowGuard);
            }
            if (low)
                product_walk<KP, ST, true>(ent, n_ent, tab, states, lane_off, vstride, nvalid, w, cur);
            const Philox4 rnd = gibbs_block(P, W.node, r, q);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                if (!((lat >> c) & 1)) continue;
                const float u = (float)(rnd.w[c] >> 8) * 0x1p-24f;
                float Z;
                cur = Q::put(cur, c, draw_kvec<KP>(w[c], K, u, Z));
                if (DEBUG) write_probs(P, W.node, r, col + c, w[c], K, Z);
            }
            Q::store(states + (int64_t)W.node * vstride + lane_off, cur);
        }
    }
}

// Debug conditionals of a table-mode node, from the product path (global tables).
template <typename ST>
__device__ void table_debug_probs(const SweepParams &P, const Work &W, int r, int64_t col,
                                  int lat, int nvalid) {
    cint32_t *d = W.d;
    const int K = d[0], KP = d[1];
    const ST *states = reinterpret_cast<const ST *>(P.states);
    const uint32_t lane_off = (uint32_t)(r * P.ld + col);
    const int64_t vstride = (int64_t)P.m * P.ld;
    const float *tab = P.table + d[3];
    typename Quad<ST>::V cur;
#define SAME_TABLE_DEBUG(KPV)                                                                   \
    {                                                                                           \
        float w[4][KPV];                                                                        \
        product_walk<KPV, ST, true>(d + d[11], d[10], tab, states, lane_off, vstride, nvalid, w,  \
                                    cur);                                                       \
        for (int c = 0; c < 4; ++c) {                                                           \
            if (!((lat >> c) & 1)) continue;                                                    \
            float Z = 0.f;                                                                      \
            for (int k = 0; k < KPV; ++k) Z += w[c][k];                                         \
            write_probs(P, W.node, r, col + c, w[c], K, Z);                                     \
        }                                                                                       \
    }
    if (KP == 2) SAME_TABLE_DEBUG(2)
    else if (KP == 4) SAME_TABLE_DEBUG(4)
    else if (KP == 8) SAME_TABLE_DEBUG(8)
    else SAME_TABLE_DEBUG(16)
#undef SAME_TABLE_DEBUG
}

// Table path: the blanket configuration indexes KT precomputed thresholds at
// cond; the drawn state is the number of thresholds at or below the 24-bit
// uniform.
template <int KT, typename ST, bool DEBUG>
__device__ void sweep_table(const SweepParams &P, const Work &W, const uint32_t *cond) {
    using Q = Quad<ST>;
    cint32_t *d = W.d;
    const int n_ent = d[8];
    cint32_t *ent = d + d[9];
    ST *states = reinterpret_cast<ST *>(P.states);
    const int64_t vstride = (int64_t)P.m * P.ld;
    for (int64_t q = W.q0 + threadIdx.x; q < W.q1; q += kBlock) {
        const int64_t col = q * 4;
        const int lat = latent_bits(P, W.node, col);
        if (!lat) continue;
        const int nvalid = P.n_cols - col < 4 ? (int)(P.n_cols - col) : 4;
        for (int r = W.r0; r < W.r1; ++r) {
            const uint32_t lane_off = (uint32_t)(r * P.ld + col);
            int idx[4] = {0, 0, 0, 0};
            typename Q::V cur;
            table_walk<ST>(ent, n_ent, states, lane_off, vstride, nvalid, idx, cur);
            const Philox4 rnd = gibbs_block(P, W.node, r, q);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                if (!((lat >> c) & 1)) continue;
                const uint32_t u24 = rnd.w[c] >> 8;
                const uint32_t *t = cond + idx[c];
                int pick = 0;
                if (KT == 1) {
                    pick = t[0] <= u24;
                } else if (KT == 2) {
                    const uint2 v = *reinterpret_cast<const uint2 *>(t);
                    pick = (v.x <= u24) + (v.y <= u24);
                } else {
#pragma unroll
                    for (int h = 0; h < KT / 4; ++h) {
                        const uint4 v = reinterpret_cast<const uint4 *>(t)[h];
                        pick += (v.x <= u24) + (v.y <= u24) + (v.z <= u24) + (v.w <= u24);
                    }
                }
                cur = Q::put(cur, c, pick);
            }
            if (DEBUG) table_debug_probs<ST>(P, W, r, col, lat, nvalid);
            Q::store(states + (int64_t)W.node * vstride + lane_off, cur);
        }
    }
}

// Main kernel: one block = one node (blockIdx.y in the launch range) x a run
// of column quads (blockIdx.x) x a range of replicas (blockIdx.z).  The
// node's mode selects the product path for KP = 2, 4, 8 or the threshold
// path.  With STAGED the block first copies its node's table (k-vector record
// or thresholds) into LDS, so every gather of the sweep is an LDS read.
template <typename ST, bool DEBUG, bool STAGED>
__global__ __launch_bounds__(kBlock) void sweep_main_kernel(SweepParams P) {
    extern __shared__ float4 lds4[];
    const Work W = block_work(P);
    cint32_t *d = W.d;
    const int mode = d[2];
    const float *tab = P.table + d[3];
    const uint32_t *cond = P.cond + d[5];
    if (STAGED) {
        if (mode == kModeTable) {
            const int len = d[6];
            uint32_t *dst = reinterpret_cast<uint32_t *>(lds4);
            for (int i = threadIdx.x; i < len; i += kBlock) dst[i] = cond[i];
            cond = dst;
        } else {
            const int len4 = d[4] >> 2;
            const float4 *src = reinterpret_cast<const float4 *>(tab);
            for (int i = threadIdx.x; i < len4; i += kBlock) lds4[i] = src[i];
            tab = reinterpret_cast<const float *>(lds4);
        }
        __syncthreads();
    }
    if (mode == kModeKP2) sweep_product<2, ST, DEBUG>(P, W, tab);
    else if (mode == kModeKP4) sweep_product<4, ST, DEBUG>(P, W, tab);
    else if (mode == kModeKP8) sweep_product<8, ST, DEBUG>(P, W, tab);
    else {
        const int KT = d[7];
        if (KT == 1) sweep_table<1, ST, DEBUG>(P, W, cond);
        else if (KT == 2) sweep_table<2, ST, DEBUG>(P, W, cond);
        else if (KT == 4) sweep_table<4, ST, DEBUG>(P, W, cond);
        else sweep_table<8, ST, DEBUG>(P, W, cond);
    }
}

// Nodes with 9 <= K <= 16 (KP = 16): kept apart because of their registers.
template <typename ST, bool DEBUG>
__global__ __launch_bounds__(kBlock) void sweep_kp16_kernel(SweepParams P) {
    const Work W = block_work(P);
    sweep_product<16, ST, DEBUG>(P, W, P.table + W.d[3]);
}

// ------------------------------------------------- generic path, K_i > 16
//
// The weight of state k is kept as (mantissa in [0.5, 1), exponent) and
// renormalised exactly after every factor, so any K fits in a few registers;
// the three passes (largest exponent, total, search) each recompute the
// products by walking the node's product-path entries for one column.

template <typename ST>
__device__ float weight_ext(cint32_t *d, const float *__restrict__ tab, const ST *__restrict__ base,
                            int64_t vstride, int c, int k, int &e) {
    using Q = Quad<ST>;
    const int n_ent = d[10];
    cint32_t *ent = d + d[11];
    int a = 0, b = 0;
    bool in_child = false;
    float mnt = 1.f;
    e = 0;
    auto factor = [&](float f) {
        mnt *= f;
        const int de = __builtin_amdgcn_frexp_expf(mnt);
        mnt = __builtin_ldexpf(mnt, -de);
        e += de;
    };
    for (int t = 0; t < n_ent; ++t) {
        const int arg = ent[3 * t + 2];
        if (arg == -3) continue;
        const int v = Q::get(Q::load(base + (int64_t)ent[3 * t] * vstride), c) * ent[3 * t + 1];
        if (arg == -1) a += v;
        else if (arg == -2) b += v;
        else {
            factor(in_child ? tab[b + k] : tab[a + k]);
            in_child = true;
            b = arg + v;
        }
    }
    factor(in_child ? tab[b + k] : tab[a + k]);
    return mnt;
}

template <typename ST, bool DEBUG>
__global__ __launch_bounds__(kBlock) void sweep_generic_kernel(SweepParams P) {
    using Q = Quad<ST>;
    const Work W = block_work(P);
    cint32_t *d = W.d;
    const int K = d[0];
    const float *tab = P.table + d[3];
    ST *states = reinterpret_cast<ST *>(P.states);
    const int64_t vstride = (int64_t)P.m * P.ld;
    for (int64_t q = W.q0 + threadIdx.x; q < W.q1; q += kBlock) {
        const int64_t col = q * 4;
        const int lat = latent_bits(P, W.node, col);
        if (!lat) continue;
        for (int r = W.r0; r < W.r1; ++r) {
            const ST *base = states + (int64_t)r * P.ld + col;
            const Philox4 rnd = gibbs_block(P, W.node, r, q);
            ST *own = states + ((int64_t)W.node * P.m + r) * P.ld + col;
            typename Q::V cur = Q::load(own);
            for (int c = 0; c < 4; ++c) {
                if (!((lat >> c) & 1)) continue;
                int E = -100000;
                for (int k = 0; k < K; ++k) {
                    int e;
                    const float mk = weight_ext<ST>(d, tab, base, vstride, c, k, e);
                    if (mk > 0.f && e > E) E = e;
                }
                float Z = 0.f;
                for (int k = 0; k < K; ++k) {
                    int e;
                    const float mk = weight_ext<ST>(d, tab, base, vstride, c, k, e);
                    Z += __builtin_ldexpf(mk, e - E);
                }
                const float t = (float)(rnd.w[c] >> 8) * 0x1p-24f * Z;
                float S = 0.f;
                int pick = -1, last_pos = 0;
                for (int k = 0; k < K; ++k) {
                    int e;
                    const float wk = __builtin_ldexpf(weight_ext<ST>(d, tab, base, vstride, c, k, e), e - E);
                    S += wk;
                    if (wk > 0.f) last_pos = k;
                    if (pick < 0 && t < S) pick = k;
                    if (DEBUG) {
                        const int64_t j = col + c;
                        if (j >= P.win_begin && j < P.win_begin + P.win)
                            P.probs[(((int64_t)W.node * P.m + r) * P.win + (j - P.win_begin)) *
                                        P.max_card + k] = wk / Z;
                    }
                }
                if (pick < 0) pick = last_pos;
                cur = Q::put(cur, c, pick);
            }
            Q::store(own, cur);
        }
    }
}

// ------------------------------------------------------ threshold tables

// One thread per blanket configuration of a table-mode node: decodes the
// configuration (blanket nodes in ascending id, last fastest), forms the log
// conditional in fp64 from max(theta, FLT_MIN), and stores the thresholds
// T_k = ceil(2^24 * S_k / Z) for k < K-1, padded with 2^24.
constexpr int kMaxBlanketTable = 24;

__global__ __launch_bounds__(kBlock) void build_thresholds_kernel(
    const int32_t *__restrict__ cprog, const int32_t *__restrict__ cprog_off,
    const int32_t *__restrict__ blk_prog, const int32_t *__restrict__ blk_first,
    const float *__restrict__ cpts, uint32_t *__restrict__ cond) {
#pragma clang fp contract(off)
    const int32_t *P = cprog + cprog_off[blk_prog[blockIdx.x]];
    const int K = P[0], KT = P[1], coff = P[2], ncfg = P[3], nbl = P[4];
    const int cfg = blk_first[blockIdx.x] + (int)threadIdx.x;
    if (cfg >= ncfg) return;
    int xb[kMaxBlanketTable];
    int rem = cfg;
    for (int t = nbl - 1; t >= 0; --t) {
        const int card = P[5 + t];
        xb[t] = rem % card;
        rem /= card;
    }
    const int32_t *q = P + 5 + nbl;
    const int own = q[0], npar = q[1];
    q += 2;
    int64_t u = 0;
    for (int j = 0; j < npar; ++j, q += 2) u += (int64_t)xb[q[0]] * q[1];
    double l[9];
    for (int k = 0; k < K; ++k)
        l[k] = log(fmax((double)cpts[own + u * K + k], (double)FLT_MIN));
    const int nch = q[0];
    ++q;
    for (int h = 0; h < nch; ++h) {
        const int offh = q[0], Kh = q[1], si = q[2], xh = xb[q[3]], ncop = q[4];
        q += 5;
        int64_t uh = 0;
        for (int j = 0; j < ncop; ++j, q += 2) uh += (int64_t)xb[q[0]] * q[1];
        for (int k = 0; k < K; ++k)
            l[k] += log(fmax((double)cpts[offh + (uh + (int64_t)k * si) * Kh + xh], (double)FLT_MIN));
    }
    double mx = l[0];
    for (int k = 1; k < K; ++k) mx = fmax(mx, l[k]);
    double S[9];
    double acc = 0.0;
    for (int k = 0; k < K; ++k) {
        acc += exp(l[k] - mx);
        S[k] = acc;
    }
    uint32_t *dst = cond + coff + (int64_t)cfg * KT;
    for (int k = 0; k < KT; ++k) {
        uint32_t t = 1u << 24;
        if (k < K - 1) {
            const double v = ceil(S[k] / acc * 16777216.0);
            t = v >= 16777216.0 ? (1u << 24) : (uint32_t)v;
        }
        dst[k] = t;
    }
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

// Histogram of (parent row, state) for one node over a run of columns and all
// m replicas.  Small CPTs (<= kRepBins bins) use kCopies interleaved LDS
// copies, lane l adding into copy l % kCopies, so lanes hitting the same bin
// rarely collide; mid-size CPTs share one LDS histogram; CPTs beyond LDS go
// straight to global atomics.  Each block flushes its non-zero bins once.
constexpr int kCopies = 32;
constexpr int kRepBins = 256;
constexpr int kLdsBins = 8192;
static_assert(kCopies * kRepBins <= kLdsBins, "LDS budget");

template <typename ST>
__global__ __launch_bounds__(kBlock) void count_kernel(const int32_t *__restrict__ cdesc,
                                                      const int32_t *__restrict__ cdesc_off,
                                                      int32_t node_base, int64_t cols_per_block,
                                                      const ST *__restrict__ states, int32_t m,
                                                      int64_t n_cols, int64_t ld,
                                                      int32_t *__restrict__ counts) {
    using Q = Quad<ST>;
    __shared__ int32_t hist[kLdsBins];
    const int node = node_base + (int)blockIdx.y;
    const int32_t *__restrict__ d = cdesc + cdesc_off[node];
    const int K = d[0], n_par = d[1], nbins = d[2], off = d[3];
    const int mode = nbins <= kRepBins ? 0 : (nbins <= kLdsBins ? 1 : 2);
    const int lds_words = mode == 0 ? nbins * kCopies : (mode == 1 ? nbins : 0);
    for (int b = threadIdx.x; b < lds_words; b += kBlock) hist[b] = 0;
    __syncthreads();
    const int copy = threadIdx.x & (kCopies - 1);
    const int64_t c0 = (int64_t)blockIdx.x * cols_per_block;
    const int64_t c1 = c0 + cols_per_block < n_cols ? c0 + cols_per_block : n_cols;
    const int64_t vstride = (int64_t)m * ld;
    for (int r = 0; r < m; ++r) {
        for (int64_t col = c0 + 4 * (int64_t)threadIdx.x; col < c1; col += 4 * kBlock) {
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
                if (col + c >= c1) break;
                const int bin = u[c] * K + Q::get(xs, c);
                if (mode == 0) atomicAdd(&hist[bin * kCopies + copy], 1);
                else if (mode == 1) atomicAdd(&hist[bin], 1);
                else atomicAdd(&counts[off + bin], 1);
            }
        }
    }
    if (mode == 2) return;
    __syncthreads();
    for (int b = threadIdx.x; b < nbins; b += kBlock) {
        int v;
        if (mode == 0) {
            v = 0;
#pragma unroll 8
            for (int k = 0; k < kCopies; ++k) v += hist[b * kCopies + ((k + b) & (kCopies - 1))];
        } else {
            v = hist[b];
        }
        if (v) atomicAdd(&counts[off + b], v);
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

template <typename ST>
void sweep_class(const SweepParams &P, int32_t klass, int32_t lds_bytes, dim3 grid,
                 hipStream_t stream) {
    const bool dbg = P.win > 0;
    const dim3 blk(dev::kBlock);
    if (klass == 0) {
        if (dbg) hipLaunchKernelGGL((dev::sweep_main_kernel<ST, true, true>), grid, blk, lds_bytes, stream, P);
        else hipLaunchKernelGGL((dev::sweep_main_kernel<ST, false, true>), grid, blk, lds_bytes, stream, P);
    } else if (klass == 1) {
        if (dbg) hipLaunchKernelGGL((dev::sweep_main_kernel<ST, true, false>), grid, blk, 0, stream, P);
        else hipLaunchKernelGGL((dev::sweep_main_kernel<ST, false, false>), grid, blk, 0, stream, P);
    } else if (klass == 2) {
        if (dbg) hipLaunchKernelGGL((dev::sweep_kp16_kernel<ST, true>), grid, blk, 0, stream, P);
        else hipLaunchKernelGGL((dev::sweep_kp16_kernel<ST, false>), grid, blk, 0, stream, P);
    } else {
        if (dbg) hipLaunchKernelGGL((dev::sweep_generic_kernel<ST, true>), grid, blk, 0, stream, P);
        else hipLaunchKernelGGL((dev::sweep_generic_kernel<ST, false>), grid, blk, 0, stream, P);
    }
}

}  // namespace

hipError_t launch_sweep(SweepParams P, int32_t begin, int32_t count, int32_t klass,
                        int32_t lds_bytes, int32_t state_bytes, hipStream_t stream) {
    if (count <= 0 || P.n_cols <= 0) return hipSuccess;
    // about 8192 blocks per launch: split the columns first, then the replicas
    const int64_t quads = (P.n_cols + 3) / 4;
    const int64_t want = (8192 + count - 1) / count;
    const int64_t max_chunks = (quads + dev::kBlock - 1) / dev::kBlock;
    int64_t chunks = want < max_chunks ? want : max_chunks;
    if (chunks < 1) chunks = 1;
    int64_t rsplit = (want + chunks - 1) / chunks;
    if (rsplit > P.m) rsplit = P.m;
    if (rsplit < 1) rsplit = 1;
    P.quads_per_block = (quads + chunks - 1) / chunks;
    P.reps_per_block = (int32_t)((P.m + rsplit - 1) / rsplit);
    const unsigned gx = (unsigned)((quads + P.quads_per_block - 1) / P.quads_per_block);
    const unsigned gz = (unsigned)((P.m + P.reps_per_block - 1) / P.reps_per_block);
    for (int32_t s = 0; s < count; s += 65535) {
        const int32_t c = count - s < 65535 ? count - s : 65535;
        P.begin = begin + s;
        dim3 grid(gx, (unsigned)c, gz);
        if (state_bytes == 1) sweep_class<int8_t>(P, klass, lds_bytes, grid, stream);
        else sweep_class<int16_t>(P, klass, lds_bytes, grid, stream);
    }
    return hipGetLastError();
}

hipError_t launch_build_thresholds(const DeviceTables &t, const float *cpts, uint32_t *cond,
                                   hipStream_t stream) {
    if (t.n_cond_blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(dev::build_thresholds_kernel, dim3(t.n_cond_blocks), dim3(dev::kBlock), 0,
                       stream, t.cprog, t.cprog_off, t.cblk_prog, t.cblk_first, cpts, cond);
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
    // about 8192 blocks in total, each a run of columns of one node (all replicas)
    const int64_t quads = (n_cols + 3) / 4;
    int64_t chunks = (8192 + n - 1) / n;
    const int64_t max_chunks = (quads + dev::kBlock - 1) / dev::kBlock;
    if (chunks > max_chunks) chunks = max_chunks;
    if (chunks < 1) chunks = 1;
    const int64_t cols_per_block = ((quads + chunks - 1) / chunks) * 4;
    const unsigned gx = (unsigned)((n_cols + cols_per_block - 1) / cols_per_block);
    for (int32_t s = 0; s < n; s += 65535) {
        const int32_t c = n - s < 65535 ? n - s : 65535;
        dim3 grid(gx, (unsigned)c, 1);
        if (state_bytes == 1)
            hipLaunchKernelGGL(dev::count_kernel<int8_t>, grid, dim3(dev::kBlock), 0, stream, t.cdesc,
                               t.cdesc_off, s, cols_per_block, (const int8_t *)states, m, n_cols, ld,
                               counts);
        else
            hipLaunchKernelGGL(dev::count_kernel<int16_t>, grid, dim3(dev::kBlock), 0, stream, t.cdesc,
                               t.cdesc_off, s, cols_per_block, (const int16_t *)states, m, n_cols, ld,
                               counts);
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
