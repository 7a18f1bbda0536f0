// gfx950 kernels of libsame: table build, colour-group Gibbs sweep, count
// histogram, moving sum, Gamma/Dirichlet resample.
//
// Data layout (HBM): states [n][m][ld] int8 (or int16), obs [n][ld] uint8.
// The fast sweep kernel works on items: one latent column of a node and a
// quad of its replicas, whose four draws take the four words of one Philox
// block; consecutive lanes take consecutive latent columns, so the state
// loads of a wavefront fall in a few cache lines per replica row.  The count
// and ingest kernels read whole column quads (dwords) per lane.
#include <hip/hip_runtime.h>
#include <type_traits>

#include <cfloat>
#include <cstdint>
#include <mutex>
#include <vector>

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
constexpr int kSweepBlock = 256;     // threads of a sweep block
constexpr int kSweepWaves = 6;       // waves per SIMD the fast sweep kernel is compiled for

// ---------------------------------------------------------------- state quads
//
// States are stored as replica quads: states[n][mq][ld][4] with mq = ceil(m/4),
// so that replica r of node i at column j is element
// ((i * mq + r / 4) * ld + j) * 4 + r % 4.  The four replicas 4 rq .. 4 rq + 3
// of one column -- a state quad, slots 0..3 -- are adjacent (4 bytes for int8,
// 8 for int16) and travel in one load or store.  Slots >= m of the last quad
// are padding.

// With 4-bit states (the Nib format) a quad is one 16-bit word, replica slot
// s in bits 4s .. 4s + 3.  Kernels address states in bytes: a node's block is
// node_bytes long and quad (rq, j) sits quad_boff bytes into it.

struct Nib {};  // tag type of the 4-bit format

// Element type of the arrays that hold single states (CSR values, targets,
// compact states): the state type, int8 for 4-bit states.
template <typename ST>
struct ElemOf {
    using T = ST;
};
template <>
struct ElemOf<Nib> {
    using T = int8_t;
};

template <typename ST>
struct Quad;

template <>
struct Quad<int8_t> {
    using V = uint32_t;
    static constexpr int kBytes = 4;
    static constexpr uint32_t kMask = 0xffu;  // one state's bits
    __device__ static V load(const int8_t *p) { return *reinterpret_cast<const uint32_t *>(p); }
    __device__ static V load_at(const char *p) { return *reinterpret_cast<const uint32_t *>(p); }
    __device__ static void store_at(char *p, V v) { *reinterpret_cast<uint32_t *>(p) = v; }
    __device__ static V load_buffer(__amdgpu_buffer_rsrc_t r, uint32_t boff) {
        return __builtin_amdgcn_raw_buffer_load_b32(r, (int)boff, 0, 0);
    }
    __device__ static void store(int8_t *p, V v) { *reinterpret_cast<uint32_t *>(p) = v; }
    __device__ static void store_buffer(__amdgpu_buffer_rsrc_t r, uint32_t boff, V v) {
        __builtin_amdgcn_raw_buffer_store_b32(v, r, (int)boff, 0, 0);
    }
    // the same state in all four slots
    __device__ static V splat(int x) { return (uint32_t)(x & 0xff) * 0x01010101u; }
    __device__ static int get(V v, int c) { return (int)((v >> (8 * c)) & 0xffu); }
    __device__ static V put(V v, int c, int x) {
        return (v & ~(0xffu << (8 * c))) | ((uint32_t)(x & 0xff) << (8 * c));
    }
    // keeps the first nvalid (1..4) slots, zeroes the rest
    __device__ static V keep(V v, int nvalid) {
        return nvalid >= 4 ? v : (v & ((1u << (8 * nvalid)) - 1u));
    }
    // the 4 states as 16-bit lanes: p[0] = slots (0, 2), p[1] = (1, 3)
    __device__ static void split(V v, uint32_t (&p)[2]) {
        p[0] = v & 0x00ff00ffu;
        p[1] = __builtin_amdgcn_perm(0u, v, 0x0c030c01u);
    }
    __device__ static constexpr int word_of(int c) { return c & 1; }
    __device__ static constexpr int half_of(int c) { return c >> 1; }
};

template <>
struct Quad<int16_t> {
    using V = uint2;
    static constexpr int kBytes = 8;
    static constexpr uint32_t kMask = 0xffffu;
    __device__ static V load(const int16_t *p) { return *reinterpret_cast<const uint2 *>(p); }
    __device__ static V load_at(const char *p) { return *reinterpret_cast<const uint2 *>(p); }
    __device__ static void store_at(char *p, V v) { *reinterpret_cast<uint2 *>(p) = v; }
    // one 8-byte load (the quad's offset is a multiple of 8 bytes)
    __device__ static V load_buffer(__amdgpu_buffer_rsrc_t r, uint32_t boff) {
        typedef uint32_t w2 __attribute__((ext_vector_type(2)));
        const w2 v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)boff, 0, 0);
        return make_uint2(v.x, v.y);
    }
    __device__ static void store(int16_t *p, V v) { *reinterpret_cast<uint2 *>(p) = v; }
    __device__ static void store_buffer(__amdgpu_buffer_rsrc_t r, uint32_t boff, V v) {
        typedef uint32_t w2 __attribute__((ext_vector_type(2)));
        const w2 x = {v.x, v.y};
        __builtin_amdgcn_raw_buffer_store_b64(x, r, (int)boff, 0, 0);
    }
    __device__ static V splat(int x) {
        const uint32_t h = (uint32_t)(x & 0xffff) * 0x10001u;
        return make_uint2(h, h);
    }
    __device__ static int get(V v, int c) {
        const uint32_t w = c < 2 ? v.x : v.y;
        return (int)((w >> (16 * (c & 1))) & 0xffffu);
    }
    __device__ static V put(V v, int c, int x) {
        const uint32_t sh = 16 * (c & 1);
        if (c < 2) v.x = (v.x & ~(0xffffu << sh)) | ((uint32_t)(x & 0xffff) << sh);
        else v.y = (v.y & ~(0xffffu << sh)) | ((uint32_t)(x & 0xffff) << sh);
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
    // the 4 states as 16-bit lanes: p[0] = slots (0, 1), p[1] = (2, 3)
    __device__ static void split(V v, uint32_t (&p)[2]) {
        p[0] = v.x;
        p[1] = v.y;
    }
    __device__ static constexpr int word_of(int c) { return c >> 1; }
    __device__ static constexpr int half_of(int c) { return c & 1; }
};

template <>
struct Quad<Nib> {
    using V = uint32_t;  // the quad in the low 16 bits
    static constexpr int kBytes = 2;
    static constexpr uint32_t kMask = 0xfu;
    __device__ static V load_at(const char *p) { return *reinterpret_cast<const uint16_t *>(p); }
    __device__ static void store_at(char *p, V v) { *reinterpret_cast<uint16_t *>(p) = (uint16_t)v; }
    __device__ static V load_buffer(__amdgpu_buffer_rsrc_t r, uint32_t boff) {
        return (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)boff, 0, 0);
    }
    __device__ static void store_buffer(__amdgpu_buffer_rsrc_t r, uint32_t boff, V v) {
        __builtin_amdgcn_raw_buffer_store_b16((uint16_t)v, r, (int)boff, 0, 0);
    }
    __device__ static V splat(int x) { return (uint32_t)(x & 0xf) * 0x1111u; }
    __device__ static int get(V v, int c) { return (int)((v >> (4 * c)) & 0xfu); }
    __device__ static V put(V v, int c, int x) {
        return (v & ~(0xfu << (4 * c))) | ((uint32_t)(x & 0xf) << (4 * c));
    }
    __device__ static V keep(V v, int nvalid) { return nvalid >= 4 ? v : (v & ((1u << (4 * nvalid)) - 1u)); }
    // the 4 states as 16-bit lanes: p[0] = slots (0, 2), p[1] = (1, 3); the
    // quad's two bytes (slots 0, 1 and slots 2, 3) first go to the two lanes
    __device__ static void split(V v, uint32_t (&p)[2]) {
        const uint32_t t = __builtin_amdgcn_perm(0u, v, 0x0c010c00u);
        p[0] = t & 0x000f000fu;
        p[1] = (t >> 4) & 0x000f000fu;
    }
    __device__ static constexpr int word_of(int c) { return c & 1; }
    __device__ static constexpr int half_of(int c) { return c >> 1; }
};

// Bytes of one node's block: mq quads of ld columns.
template <typename ST>
__device__ __forceinline__ int64_t node_bytes(int32_t m, int64_t ld) {
    return (int64_t)((m + 3) >> 2) * ld * Quad<ST>::kBytes;
}

// Byte offset of quad rq at column j inside a node's block.
template <typename ST>
__device__ __forceinline__ uint32_t quad_boff(int rq, int64_t ld, int64_t j) {
    return (uint32_t)(((int64_t)rq * ld + j) * Quad<ST>::kBytes);
}

// ---------------------------------------------------------------- entry walks

// Two 16-bit lanes per 32-bit word: v_pk_mad_u16 computes a * b + c in both.
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pk_mad_u16(uint32_t a, uint32_t b, uint32_t c) {
    const u16x2 r = __builtin_bit_cast(u16x2, a) * __builtin_bit_cast(u16x2, b) +
                    __builtin_bit_cast(u16x2, c);
    return __builtin_bit_cast(uint32_t, r);
}

// LDS bytes (address space 3: ds_read instructions, not flat loads).
typedef const __attribute__((address_space(3))) char lds_char;

// Buffer resource over n_bytes at base (uniform): raw buffer loads take a
// 32-bit vector byte offset, with no 64-bit address arithmetic per lane, and
// any offset at or past n_bytes reads 0 instead of touching memory.
constexpr int32_t kBufferWord3 = 0x00020000;  // 32-bit data format, no swizzle

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void *base, uint32_t n_bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)n_bytes,
                                             kBufferWord3);
}

// State quad of node `node` (its block of nbytes bytes, under 2^31) at the
// lane's byte offset.
template <typename ST>
__device__ __forceinline__ typename Quad<ST>::V load_row(const void *__restrict__ states, int32_t node,
                                                         int64_t nbytes, uint32_t lane_boff) {
    const __amdgpu_buffer_rsrc_t r =
        buffer_rsrc(reinterpret_cast<const char *>(states) + (uint64_t)(uint32_t)node * (uint32_t)nbytes,
                    (uint32_t)nbytes);
    return Quad<ST>::load_buffer(r, lane_boff);
}

constexpr int kEntryBatch = 8;  // most state rows in flight per batch

// Loads the state quads of the N entries (node, mult) at e, all before the
// first use, and hands each to f with its multiplier.
template <int N, typename ST, typename F>
__device__ __forceinline__ void entry_batch(cint32_t *e, const void *__restrict__ states,
                                            int64_t vstride, uint32_t lane_boff, F &f) {
    typename Quad<ST>::V s[N];
#pragma unroll
    for (int t = 0; t < N; ++t) s[t] = load_row<ST>(states, e[2 * t], vstride, lane_boff);
#pragma unroll
    for (int t = 0; t < N; ++t) f(s[t], (uint32_t)e[2 * t + 1]);
}

// Walks the n_e entries at e in batches of at most kEntryBatch.  n_e is
// uniform, so the size switch is a scalar branch and no slot is wasted.
template <typename ST, typename F>
__device__ __forceinline__ void walk_entries(cint32_t *e, int n_e, const void *__restrict__ states,
                                             int64_t vstride, uint32_t lane_boff, F &f) {
    for (; n_e > 0; n_e -= kEntryBatch, e += 2 * kEntryBatch) {
        switch (n_e < kEntryBatch ? n_e : kEntryBatch) {
        case 1: entry_batch<1, ST>(e, states, vstride, lane_boff, f); break;
        case 2: entry_batch<2, ST>(e, states, vstride, lane_boff, f); break;
        case 3: entry_batch<3, ST>(e, states, vstride, lane_boff, f); break;
        case 4: entry_batch<4, ST>(e, states, vstride, lane_boff, f); break;
        case 5: entry_batch<5, ST>(e, states, vstride, lane_boff, f); break;
        case 6: entry_batch<6, ST>(e, states, vstride, lane_boff, f); break;
        case 7: entry_batch<7, ST>(e, states, vstride, lane_boff, f); break;
        default: entry_batch<8, ST>(e, states, vstride, lane_boff, f); break;
        }
    }
}

// 16-bit lane c of a packed index pair (lane layout in Quad<ST>::split).
template <typename ST>
__device__ __forceinline__ uint32_t packed_index(const uint32_t (&Pk)[2], int c) {
    const uint32_t v = Pk[Quad<ST>::word_of(c)];
    return Quad<ST>::half_of(c) ? v >> 16 : v & 0xffffu;
}

// ---------------------------------------------------------------- k-vectors

// Reads KP floats at p (8-byte aligned for KP == 2 or 6, 16-byte otherwise).
template <int KP, typename PTR>
__device__ __forceinline__ void read_kvec(PTR p, float (&f)[KP]) {
    if (KP == 2 || KP == 6) {
#pragma unroll
        for (int q = 0; q < KP / 2; ++q) {
            const float2 v = reinterpret_cast<const float2 *>(p)[q];
            f[2 * q] = v.x;
            f[2 * q + 1] = v.y;
        }
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

// Native vector types (HIP's float4 class cannot be read from LDS lvalues).
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int KP>
__device__ __forceinline__ void read_kvec_lds(lds_char *p, float (&f)[KP]) {
    typedef const __attribute__((address_space(3))) f32x2 lf2;
    typedef const __attribute__((address_space(3))) f32x4 lf4;
    if (KP == 2 || KP == 6) {
#pragma unroll
        for (int q = 0; q < KP / 2; ++q) {
            const f32x2 v = reinterpret_cast<lf2 *>(p)[q];
            f[2 * q] = v.x;
            f[2 * q + 1] = v.y;
        }
        return;
    }
#pragma unroll
    for (int q = 0; q < KP / 4; ++q) {
        const f32x4 v = reinterpret_cast<lf4 *>(p)[q];
        f[4 * q + 0] = v.x;
        f[4 * q + 1] = v.y;
        f[4 * q + 2] = v.z;
        f[4 * q + 3] = v.w;
    }
}

constexpr int log2i(int v) { return v <= 1 ? 0 : 1 + log2i(v / 2); }

// Global-memory bytes (address space 1) from a scalar base: with a scalar
// base and a 32-bit vector offset computed in the same block, the loads take
// the scalar-base form (no 64-bit vector address arithmetic).
typedef const __attribute__((address_space(1))) char global_char;

__device__ __forceinline__ global_char *scalar_global_ptr(const void *p) {
    const uint64_t a = reinterpret_cast<uint64_t>(p);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    return reinterpret_cast<global_char *>(((uint64_t)hi << 32) | lo);
}

template <int KP>
__device__ __forceinline__ void read_kvec_global(global_char *p, float (&f)[KP]) {
    typedef const __attribute__((address_space(1))) f32x2 gf2;
    typedef const __attribute__((address_space(1))) f32x4 gf4;
    if (KP == 2 || KP == 6) {
#pragma unroll
        for (int q = 0; q < KP / 2; ++q) {
            const f32x2 v = reinterpret_cast<gf2 *>(p)[q];
            f[2 * q] = v.x;
            f[2 * q + 1] = v.y;
        }
        return;
    }
#pragma unroll
    for (int q = 0; q < KP / 4; ++q) {
        const f32x4 v = reinterpret_cast<gf4 *>(p)[q];
        f[4 * q + 0] = v.x;
        f[4 * q + 1] = v.y;
        f[4 * q + 2] = v.z;
        f[4 * q + 3] = v.w;
    }
}

// Unit of a global fast-list index: one k-vector (KP floats), or 8 bytes for
// KP = 6, whose 24-byte k-vectors do not divide the records' 64-byte group
// alignment.
template <int KP>
constexpr int kvec_unit_shift() { return KP == 6 ? 3 : log2i(4 * KP); }

// The k-vector at packed index idx: a byte offset into the staged record
// (STAGED) or an index in kvec_unit_shift units into the node's global record.
template <int KP, bool STAGED>
__device__ __forceinline__ void fast_kvec(lds_char *lds, global_char *gtab, uint32_t idx, float (&f)[KP]) {
    if (STAGED) read_kvec_lds<KP>(lds + idx, f);
    else read_kvec_global<KP>(gtab + (idx << kvec_unit_shift<KP>()), f);
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

// Same conditional from the wide list (32-bit float offsets, any record
// size) for the four slots of a state quad: wide kernel, table-mode debug
// output.  Slots >= nvalid read their states as 0.
template <int KP, typename ST, bool RESCALE>
__device__ __forceinline__ void wide_product(cint32_t *g, int n_groups, const float *__restrict__ tab,
                                             const void *__restrict__ states, int64_t vstride,
                                             uint32_t lane_boff, int nvalid, float (&w)[4][KP]) {
    using Q = Quad<ST>;
    for (int j = 0; j < n_groups; ++j) {
        const int n_e = g[0];
        uint32_t idx[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) idx[c] = (uint32_t)g[1];
        auto acc = [&](typename Q::V v, uint32_t mult) {
            v = Q::keep(v, nvalid);
#pragma unroll
            for (int c = 0; c < 4; ++c) idx[c] += (uint32_t)Q::get(v, c) * mult;
        };
        walk_entries<ST>(g + 2, n_e, states, vstride, lane_boff, acc);
        g += 2 + 2 * n_e;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            float f[KP];
            read_kvec<KP>(tab + idx[c], f);
            if (j == 0) {
#pragma unroll
                for (int k = 0; k < KP; ++k) w[c][k] = f[k];
            } else {
#pragma unroll
                for (int k = 0; k < KP; ++k) w[c][k] *= f[k];
            }
            if (RESCALE) renorm<KP>(w[c]);
        }
    }
}

// ---------------------------------------------------------------- draws

// In-place running sums S_k = w_0 + ... + w_k.
template <int KP>
__device__ __forceinline__ void running_sums(float (&w)[KP]) {
#pragma unroll
    for (int k = 1; k < KP; ++k) w[k] += w[k - 1];
}

// Inverse-CDF draw from running sums S (entries K..KP-1 repeat Z = S_{K-1}):
// the smallest k with u*Z < S_k, i.e. the number of S_k <= u*Z.  When
// rounding makes u*Z reach Z, the largest k whose weight is positive (whose
// running sum grows) is taken.
template <int KP>
__device__ __forceinline__ int draw_sums(const float (&S)[KP], int K, float u) {
    const float t = u * S[KP - 1];
    int pick = 0;
#pragma unroll
    for (int k = 0; k < KP; ++k) pick += (S[k] <= t) ? 1 : 0;
    if (pick >= K) {
        pick = 0;
#pragma unroll
        for (int k = 1; k < KP; ++k)
            if (k < K && S[k] > S[k - 1]) pick = k;
    }
    return pick;
}

// Z below this sends the quad through the renormalising walk: Z >= 2^-96
// keeps the largest weight (>= Z / 16) at or above 2^-100.
constexpr float kUnderflowZ = 0x1p-96f;

// ---------------------------------------------------------------- block work

// The block's share of the work: a run of column quads of one node and a
// range of replicas.
struct Work {
    int node;
    cint32_t *d;
    int64_t q0, q1;
    int r0, r1;
};

// Blocks are dealt to the XCDs round robin by linear block id.  The 1-D grid
// is decoded so that the blocks one XCD receives in order take every node of
// the launch for one slab (column chunk x replica range) before the next
// slab: the blocks resident on an XCD then read the same columns of the
// shared blanket rows, which stay in that XCD's L2.
constexpr uint32_t kXcds = 8;
constexpr int kSweepQuadsPerLane = 1;  // column quads per lane in one sweep block
constexpr int kMinSweepBlocks = 4096;  // replicas are split below this many blocks
constexpr int64_t kMinSweepQuads = 64;  // narrowest column chunk of a fast sweep block (quads)
constexpr int kCountQuadsPerLane = 8;  // adjacent columns (state quads) per lane and iteration of a count block

__device__ __forceinline__ void decode_block(uint32_t b, uint32_t count, uint32_t &local,
                                             int64_t &slab) {
    const uint32_t xcd = b % kXcds, j = b / kXcds;
    local = j % count;
    slab = (int64_t)(j / count) * kXcds + xcd;
}

__device__ __forceinline__ Work block_work(const SweepParams &P) {
    uint32_t local;
    int64_t slab;
    decode_block(blockIdx.x, (uint32_t)P.count, local, slab);
    Work w;
    w.node = as_const(P.order)[P.begin + (int32_t)local];
    w.d = as_const(P.desc) + as_const(P.desc_off)[w.node];
    if (slab >= P.n_slabs) {  // padding block of the last round
        w.q0 = w.q1 = 0;
        w.r0 = w.r1 = 0;
        return w;
    }
    // consecutive colour launches walk the columns in opposite directions, so
    // that a launch starts on the columns the previous one touched last (still
    // in the memory-side cache)
    if (P.reverse) slab = P.n_slabs - 1 - slab;
    const int64_t chunk = slab / P.rsplit;
    const int rpart = (int)(slab % P.rsplit);
    const int64_t nquads = (P.n_cols + 3) >> 2;
    w.q0 = chunk * P.quads_per_block;
    w.q1 = w.q0 + P.quads_per_block < nquads ? w.q0 + P.quads_per_block : nquads;
    w.r0 = rpart * P.reps_per_block;
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

// The Philox block of the Gibbs draws of node `node`, minibatch column j and
// the replica quad 4 rq .. 4 rq + 3: counter {g, node, rq, sweep} with g =
// col_offset + j the global column; word c is replica 4 rq + c's uniform.
__device__ __forceinline__ Philox4 gibbs_block(const SweepParams &P, int node, int rq, int64_t j) {
    return philox4x32_10((uint32_t)(P.col_offset + j), (uint32_t)node, (uint32_t)rq, P.sweep_id, P.key0,
                         P.key1);
}

__device__ __forceinline__ float uniform24(uint32_t word) { return (float)(word >> 8) * 0x1p-24f; }

// ------------------------------------------------------- sweep items
//
// The fast kernel's unit of work is an item: one latent column j of the
// block's column chunk and a quad of replicas 4 rq .. 4 rq + 3 (fewer at the
// end of the replica range).  All four draws of an item are latent -- the
// obs mask is shared by the replicas -- so no lane computes a conditional
// that nobody draws, and one Philox block gives the item's four uniforms.
// The item's four states of any blanket node are one state quad (4 or 8
// bytes at quad_boff(rq, j)), read with one load and split into two words of
// 16-bit lanes (Quad<ST>::split) for the v_pk_mad_u16 index arithmetic.
// Padding slots of a partial quad (replicas >= m) are masked to state 0
// before use, so every index stays inside the node's tables whatever they
// hold; the item's store writes their draws back (valid states).

// Buffer resource over node `node`'s state quads (offsets past them read 0).
// (node >= 0 and nbytes < 2^31: a 32 x 32 -> 64-bit product)
template <typename ST>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t node_rsrc(const void *states, int32_t node, int64_t nbytes) {
    return buffer_rsrc(reinterpret_cast<const char *>(states) + (uint64_t)(uint32_t)node * (uint32_t)nbytes,
                       (uint32_t)nbytes);
}

constexpr int kItemBatch = 4;  // blanket entries whose state quads are in flight together
constexpr int kFlatGroups = 4;  // product nodes with this many groups take the flat entry walk

// Adds the N entries (node, mult) at e to the item's packed index: every
// entry's state quad is loaded before the first is used; slots >= nrep read 0.
template <int N, typename ST>
__device__ __forceinline__ void item_entries(cint32_t *e, const void *__restrict__ states, int64_t vstride,
                                             uint32_t qoff, int nrep, uint32_t (&Pk)[2]) {
    using Q = Quad<ST>;
    typename Q::V v[N];
#pragma unroll
    for (int t = 0; t < N; ++t) v[t] = Q::load_buffer(node_rsrc<ST>(states, e[2 * t], vstride), qoff);
#pragma unroll
    for (int t = 0; t < N; ++t) {
        const uint32_t mult = (uint32_t)e[2 * t + 1];
        uint32_t p[2];
        Q::split(Q::keep(v[t], nrep), p);
        Pk[0] = pk_mad_u16(p[0], mult, Pk[0]);
        Pk[1] = pk_mad_u16(p[1], mult, Pk[1]);
    }
}

// Packed index of one group of a fast list for an item; advances g.  The
// scheduling barrier keeps the compiler from hoisting the next group's loads
// above this group's use of its own (which needs more registers than the
// occupancy bound allows).
template <typename ST>
__device__ __forceinline__ void item_group(cint32_t *&g, const void *__restrict__ states, int64_t vstride,
                                           uint32_t qoff, int nrep, uint32_t (&Pk)[2]) {
    __builtin_amdgcn_sched_barrier(0);
    int n_e = g[0];
    Pk[0] = Pk[1] = (uint32_t)g[1];
    cint32_t *e = g + 2;
    g += 2 + 2 * n_e;
    for (; n_e > 0; n_e -= kItemBatch, e += 2 * kItemBatch) {
        switch (n_e < kItemBatch ? n_e : kItemBatch) {
        case 1: item_entries<1, ST>(e, states, vstride, qoff, nrep, Pk); break;
        case 2: item_entries<2, ST>(e, states, vstride, qoff, nrep, Pk); break;
        case 3: item_entries<3, ST>(e, states, vstride, qoff, nrep, Pk); break;
        default: item_entries<4, ST>(e, states, vstride, qoff, nrep, Pk); break;
        }
    }
}

// Multiplies the k-vectors of a group into the four slots' weights (from LDS
// when FROM_LDS, else from global memory); FIRST: the group's k-vectors are
// the weights (the product of one factor).
template <int KP, typename ST, bool FROM_LDS, bool RESCALE, bool FIRST = false>
__device__ __forceinline__ void item_multiply(lds_char *lds, global_char *gtab, const uint32_t (&Pk)[2],
                                              float (&w)[4][KP]) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        float f[KP];
        fast_kvec<KP, FROM_LDS>(lds, gtab, packed_index<ST>(Pk, c), f);
#pragma unroll
        for (int k = 0; k < KP; ++k) w[c][k] = FIRST ? f[k] : w[c][k] * f[k];
        if (RESCALE) renorm<KP>(w[c]);
    }
}

// Unnormalised full conditional (Sec. 4: own CPT entry times the children's
// entries) of the item's four replica slots from a fast product list: the
// first n_staged groups read their k-vectors from the LDS copy of the record
// (byte indices), the others from global memory (k-vector units).  The
// list's first group (every list has one) gives the weights; each later group
// multiplies into them, in list order.  With RESCALE every running product is renormalised
// after each factor, which keeps it away from fp32 underflow.
template <int KP, typename ST, bool STAGED, bool RESCALE>
__device__ __forceinline__ void item_product(cint32_t *g, int n_groups, int n_staged, lds_char *lds,
                                             global_char *gtab, const void *__restrict__ states, int64_t vstride,
                                             uint32_t qoff, int nrep, float (&w)[4][KP]) {
    uint32_t Pk[2];
    item_group<ST>(g, states, vstride, qoff, nrep, Pk);
    if (STAGED && n_staged > 0) item_multiply<KP, ST, true, RESCALE, true>(lds, gtab, Pk, w);
    else item_multiply<KP, ST, false, RESCALE, true>(lds, gtab, Pk, w);
    // the staged groups, then the global ones: two loops, so that each keeps
    // only its own addressing live
    int j = 1;
    if (STAGED) {
        for (; j < n_staged; ++j) {
            item_group<ST>(g, states, vstride, qoff, nrep, Pk);
            item_multiply<KP, ST, true, RESCALE>(lds, gtab, Pk, w);
        }
    }
    for (; j < n_groups; ++j) {
        item_group<ST>(g, states, vstride, qoff, nrep, Pk);
        item_multiply<KP, ST, false, RESCALE>(lds, gtab, Pk, w);
    }
}

// The n entries of a flat batch at e (4 words each): every entry's state
// quad is loaded before the first use.
template <int N, typename ST, int NB>
__device__ __forceinline__ void flat_loads(cint32_t *e, const void *__restrict__ states, int64_t vstride,
                                           uint32_t qoff, typename Quad<ST>::V (&v)[NB]) {
#pragma unroll
    for (int t = 0; t < N; ++t) v[t] = Quad<ST>::load_buffer(node_rsrc<ST>(states, e[4 * t], vstride), qoff);
}

// The product over a node's flat entry list (every group's k-vectors from
// LDS when FROM_LDS, else from global memory): entries are loaded in batches
// (of kItemBatch, twice that for two-state nodes) across group boundaries,
// and a group's factor is applied as soon as its last entry has been added.
// The weights start at one (exact).
template <int KP, typename ST, bool FROM_LDS>
__device__ __forceinline__ void item_product_flat(cint32_t *f, lds_char *lds, global_char *gtab,
                                                  const void *__restrict__ states, int64_t vstride, uint32_t qoff,
                                                  int nrep, float (&w)[4][KP]) {
    using Q = Quad<ST>;
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int k = 0; k < KP; ++k) w[c][k] = 1.f;
    const int E = f[0];
    cint32_t *e = f + 4;
    uint32_t Pk[2] = {0u, 0u};
    // two-state nodes keep twice as many entries in flight (few registers)
    constexpr int NB = KP <= 2 ? 2 * kItemBatch : kItemBatch;
    for (int b = 0; b < E; b += NB, e += 4 * NB) {
        __builtin_amdgcn_sched_barrier(0);
        const int n = E - b < NB ? E - b : NB;
        typename Q::V v[NB];
        switch (n) {
        case 1: flat_loads<1, ST, NB>(e, states, vstride, qoff, v); break;
        case 2: flat_loads<2, ST, NB>(e, states, vstride, qoff, v); break;
        case 3: flat_loads<3, ST, NB>(e, states, vstride, qoff, v); break;
        case 4: flat_loads<4, ST, NB>(e, states, vstride, qoff, v); break;
        case 5: flat_loads<NB >= 5 ? 5 : 4, ST, NB>(e, states, vstride, qoff, v); break;
        case 6: flat_loads<NB >= 6 ? 6 : 4, ST, NB>(e, states, vstride, qoff, v); break;
        case 7: flat_loads<NB >= 7 ? 7 : 4, ST, NB>(e, states, vstride, qoff, v); break;
        default: flat_loads<NB, ST, NB>(e, states, vstride, qoff, v); break;
        }
#pragma unroll
        for (int s = 0; s < NB; ++s) {
            if (s >= n) break;  // uniform
            __builtin_amdgcn_sched_barrier(0);
            cint32_t *x = e + 4 * s;
            const int flags = x[3];
            if (flags & 1) Pk[0] = Pk[1] = (uint32_t)x[2];
            uint32_t p[2];
            Q::split(Q::keep(v[s], nrep), p);
            Pk[0] = pk_mad_u16(p[0], (uint32_t)x[1], Pk[0]);
            Pk[1] = pk_mad_u16(p[1], (uint32_t)x[1], Pk[1]);
            if (flags & 2) item_multiply<KP, ST, FROM_LDS, false>(lds, gtab, Pk, w);
        }
    }
}

// The block's latent columns and its replica range, as items.
struct Items {
    const uint16_t *col;  // latent columns of the chunk, as offsets from c0 (LDS)
    int64_t c0;
    int ncl, nrq, r0, r1;
    float inv;            // 1 / ncl
};

// Item t -> (column j, first replica rb, replicas nrep).
__device__ __forceinline__ void item_of(const Items &I, int t, int64_t &j, int &rb, int &nrep) {
    int rq = (int)((float)t * I.inv);  // t, ncl < 2^24: off by at most one
    int k = t - rq * I.ncl;
    if (k < 0) {
        --rq;
        k += I.ncl;
    } else if (k >= I.ncl) {
        ++rq;
        k -= I.ncl;
    }
    j = I.c0 + I.col[k];
    rb = I.r0 + 4 * rq;
    nrep = I.r1 - rb < 4 ? I.r1 - rb : 4;
}

// Product path (classes 0 and 1, KP <= 8): the block's items, one per lane
// at a time.
template <int KP, typename ST, bool DEBUG, bool STAGED>
__device__ __forceinline__ void sweep_product(const SweepParams &P, const Work &W, const Items &I, lds_char *lds,
                                              global_char *gtab) {
    cint32_t *d = W.d;
    const int K = d[0], n_groups = d[8], n_staged = STAGED ? d[13] : 0;
    cint32_t *grp = d + d[9];
    char *states = reinterpret_cast<char *>(P.states);
    const int64_t vstride = node_bytes<ST>(P.m, P.ld);
    const __amdgpu_buffer_rsrc_t own = node_rsrc<ST>(states, W.node, vstride);
    const int n_items = I.ncl * I.nrq;
    for (int t = threadIdx.x; t < n_items; t += kSweepBlock) {
        int64_t j;
        int rb, nrep;
        item_of(I, t, j, rb, nrep);
        const uint32_t qoff = quad_boff<ST>(rb >> 2, P.ld, j);
        float w[4][KP];
        // nodes with many groups (all from LDS, or all from global memory)
        // walk their flat entry list: fewer dependent loads per item
        if (n_groups < kFlatGroups || (STAGED && n_staged != n_groups))
            item_product<KP, ST, STAGED, false>(grp, n_groups, n_staged, lds, gtab, states, vstride, qoff, nrep, w);
        else if (!STAGED)
            item_product_flat<KP, ST, false>(d + d[15], lds, gtab, states, vstride, qoff, nrep, w);
        else
            item_product_flat<KP, ST, true>(d + d[15], lds, gtab, states, vstride, qoff, nrep, w);
        float wd[4][KP];
        if (DEBUG) {
#pragma unroll
            for (int c = 0; c < 4; ++c)
#pragma unroll
                for (int k = 0; k < KP; ++k) wd[c][k] = w[c][k];
        }
        bool low = false;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            running_sums<KP>(w[c]);
            low |= c < nrep && !(w[c][KP - 1] >= kUnderflowZ);
        }
        if (low) {
            item_product<KP, ST, STAGED, true>(grp, n_groups, n_staged, lds, gtab, states, vstride, qoff, nrep, w);
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                if (DEBUG) {
#pragma unroll
                    for (int k = 0; k < KP; ++k) wd[c][k] = w[c][k];
                }
                running_sums<KP>(w[c]);
            }
        }
        const Philox4 rnd = gibbs_block(P, W.node, rb >> 2, j);
        typename Quad<ST>::V out{};
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            out = Quad<ST>::put(out, c, draw_sums<KP>(w[c], K, uniform24(rnd.w[c])));
            if (DEBUG && c < nrep) write_probs(P, W.node, rb + c, j, wd[c], K, w[c][KP - 1]);
        }
        Quad<ST>::store_buffer(own, qoff, out);
    }
}

// Debug conditional of a table-mode node for replica r and column j, from
// its wide list (global tables): the product over the state quad that holds
// replica r, of which slot r % 4 is written out.
template <typename ST>
__device__ void table_debug_prob(const SweepParams &P, const Work &W, int r, int64_t j) {
    cint32_t *d = W.d;
    const int K = d[0], KP = d[1];
    const char *states = reinterpret_cast<const char *>(P.states);
    const int rb = r & ~3;
    const int nvalid = P.m - rb < 4 ? P.m - rb : 4;
    const int c = r & 3;
    const uint32_t lane_boff = quad_boff<ST>(rb >> 2, P.ld, j);
    const int64_t vstride = node_bytes<ST>(P.m, P.ld);
    const float *tab = P.table + d[3];
#define SAME_TABLE_DEBUG(KPV)                                                                     \
    {                                                                                             \
        float w[4][KPV];                                                                          \
        wide_product<KPV, ST, true>(d + d[11], d[10], tab, states, vstride, lane_boff, nvalid, w); \
        float Z = 0.f;                                                                            \
        for (int k = 0; k < KPV; ++k) Z += w[c][k];                                               \
        write_probs(P, W.node, r, j, w[c], K, Z);                                                 \
    }
    if (KP == 2) SAME_TABLE_DEBUG(2)
    else if (KP == 4) SAME_TABLE_DEBUG(4)
    else if (KP == 6) SAME_TABLE_DEBUG(6)
    else if (KP == 8) SAME_TABLE_DEBUG(8)
    else SAME_TABLE_DEBUG(16)
#undef SAME_TABLE_DEBUG
}

// KT thresholds of a blanket configuration: the row at byte offset idx of the
// staged table (LDS) or row idx of the table in global memory.
template <int KT>
__device__ __forceinline__ void read_thresholds(bool from_lds, lds_char *lds, global_char *gcond, uint32_t idx,
                                                uint32_t (&th)[KT]) {
    if (from_lds) {
        typedef const __attribute__((address_space(3))) uint32_t lu32;
        typedef const __attribute__((address_space(3))) u32x2 lu2;
        typedef const __attribute__((address_space(3))) u32x4 lu4;
        lds_char *p = lds + idx;
        if (KT == 1) {
            th[0] = *reinterpret_cast<lu32 *>(p);
        } else if (KT == 2) {
            const u32x2 v = *reinterpret_cast<lu2 *>(p);
            th[0] = v.x;
            th[1] = v.y;
        } else {
#pragma unroll
            for (int h = 0; h < KT / 4; ++h) {
                const u32x4 v = reinterpret_cast<lu4 *>(p)[h];
                th[4 * h] = v.x;
                th[4 * h + 1] = v.y;
                th[4 * h + 2] = v.z;
                th[4 * h + 3] = v.w;
            }
        }
    } else {
        typedef const __attribute__((address_space(1))) uint32_t gu32;
        typedef const __attribute__((address_space(1))) u32x2 gu2;
        typedef const __attribute__((address_space(1))) u32x4 gu4;
        global_char *p = gcond + (idx << log2i(4 * KT));
        if (KT == 1) {
            th[0] = *reinterpret_cast<gu32 *>(p);
        } else if (KT == 2) {
            const u32x2 v = *reinterpret_cast<gu2 *>(p);
            th[0] = v.x;
            th[1] = v.y;
        } else {
#pragma unroll
            for (int h = 0; h < KT / 4; ++h) {
                const u32x4 v = reinterpret_cast<gu4 *>(p)[h];
                th[4 * h] = v.x;
                th[4 * h + 1] = v.y;
                th[4 * h + 2] = v.z;
                th[4 * h + 3] = v.w;
            }
        }
    }
}

// Threshold path (classes 0 and 1): the blanket configuration of each
// replica slot selects KT thresholds; the drawn state is the number of them
// at or below the 24-bit uniform.
template <int KT, typename ST, bool DEBUG, bool STAGED>
__device__ __forceinline__ void sweep_table(const SweepParams &P, const Work &W, const Items &I, lds_char *lds,
                                            global_char *gcond) {
    cint32_t *d = W.d;
    cint32_t *grp = d + d[9];
    const bool tab_lds = STAGED && d[13] > 0;  // uniform: thresholds staged in LDS
    char *states = reinterpret_cast<char *>(P.states);
    const int64_t vstride = node_bytes<ST>(P.m, P.ld);
    const __amdgpu_buffer_rsrc_t own = node_rsrc<ST>(states, W.node, vstride);
    const int n_items = I.ncl * I.nrq;
    for (int t = threadIdx.x; t < n_items; t += kSweepBlock) {
        int64_t j;
        int rb, nrep;
        item_of(I, t, j, rb, nrep);
        const uint32_t qoff = quad_boff<ST>(rb >> 2, P.ld, j);
        cint32_t *g = grp;
        uint32_t Pk[2];
        item_group<ST>(g, states, vstride, qoff, nrep, Pk);
        const Philox4 rnd = gibbs_block(P, W.node, rb >> 2, j);
        typename Quad<ST>::V out{};
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const uint32_t u24 = rnd.w[c] >> 8;
            uint32_t th[KT];
            read_thresholds<KT>(tab_lds, lds, gcond, packed_index<ST>(Pk, c), th);
            int pick = 0;
#pragma unroll
            for (int k = 0; k < KT; ++k) pick += th[k] <= u24 ? 1 : 0;
            out = Quad<ST>::put(out, c, pick);
        }
        Quad<ST>::store_buffer(own, qoff, out);
        if (DEBUG) {
            for (int c = 0; c < nrep; ++c) table_debug_prob<ST>(P, W, rb + c, j);
        }
    }
}

// Fast kernel: one block = one node x a chunk of columns x a range of
// replicas (block_work).  The block first lists the chunk's latent columns
// of its node in LDS (a block-wide prefix sum over the lanes' obs words) and,
// with STAGED, copies the staged part of its node's table record (the whole
// record of a class-0 node: k-vectors or thresholds; the smallest k-vector
// groups of a larger record) into LDS; then its lanes take the items
// (latent column, replica quad) in turn.  The node's mode selects the
// product path for KP = 2, 4, 6, 8 or the threshold path.
// At least kSweepWaves waves per SIMD (the debug variant keeps the default
// bound).
template <typename ST, bool DEBUG, bool STAGED>
__global__ __launch_bounds__(kSweepBlock, DEBUG ? 1 : kSweepWaves) void sweep_fast_kernel(SweepParams P) {
    if (P.ids) P.sweep_id = P.ids[0];
    extern __shared__ float4 lds4[];
    __shared__ uint16_t lcol[4 * kSweepBlock];
    __shared__ int32_t wave_n[kSweepBlock / 64];
    const Work W = block_work(P);
    if (W.q0 >= W.q1) return;  // uniform across the block
    cint32_t *d = W.d;
    const int mode = d[2];
    const float *tab = P.table + d[3];
    const uint32_t *cond = P.cond + d[5];
    // latent columns of the chunk: lane l reads the obs word of columns
    // c0 + 4l .. c0 + 4l + 3
    const int64_t c0 = W.q0 * 4;
    const int64_t col = c0 + 4 * (int64_t)threadIdx.x;
    const int lat = col < W.q1 * 4 ? latent_bits(P, W.node, col) : 0;
    const int cnt = __builtin_popcount(lat);
    const uint64_t b0 = __ballot(cnt & 1), b1 = __ballot(cnt & 2), b2 = __ballot(cnt & 4);
    auto below = [](uint64_t b) {  // set lanes below this one
        return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0u));
    };
    const int pre = below(b0) + 2 * below(b1) + 4 * below(b2);
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0)
        wave_n[wave] = __builtin_popcountll(b0) + 2 * __builtin_popcountll(b1) + 4 * __builtin_popcountll(b2);
    if (STAGED) {
        const float4 *src = reinterpret_cast<const float4 *>(mode == kModeTable ? (const void *)cond
                                                                                : (const void *)tab);
        const int len4 = d[14] >> 2;
        for (int i = threadIdx.x; i < len4; i += kSweepBlock) lds4[i] = src[i];
    }
    __syncthreads();
    int base = 0, ncl = 0;
#pragma unroll
    for (int v = 0; v < kSweepBlock / 64; ++v) {
        const int nv = wave_n[v];
        base += v < wave ? nv : 0;
        ncl += nv;
    }
    int pos = base + pre;
#pragma unroll
    for (int c = 0; c < 4; ++c)
        if ((lat >> c) & 1) lcol[pos++] = (uint16_t)(4 * threadIdx.x + c);
    __syncthreads();
    if (ncl == 0) return;  // uniform
    Items I;
    I.col = lcol;
    I.c0 = c0;
    I.ncl = ncl;
    I.r0 = W.r0;
    I.r1 = W.r1;
    I.nrq = (W.r1 - W.r0 + 3) >> 2;
    I.inv = 1.f / (float)ncl;
    lds_char *lds = (lds_char *)lds4;
    global_char *gt = scalar_global_ptr(tab);
    if (mode == kModeKP2) sweep_product<2, ST, DEBUG, STAGED>(P, W, I, lds, gt);
    else if (mode == kModeKP4) sweep_product<4, ST, DEBUG, STAGED>(P, W, I, lds, gt);
    else if (mode == kModeKP6) sweep_product<6, ST, DEBUG, STAGED>(P, W, I, lds, gt);
    else if (mode == kModeKP8) sweep_product<8, ST, DEBUG, STAGED>(P, W, I, lds, gt);
    else {
        const int KT = d[7];
        global_char *gc = scalar_global_ptr(cond);
        if (KT == 1) sweep_table<1, ST, DEBUG, STAGED>(P, W, I, lds, gc);
        else if (KT == 2) sweep_table<2, ST, DEBUG, STAGED>(P, W, I, lds, gc);
        else if (KT == 4) sweep_table<4, ST, DEBUG, STAGED>(P, W, I, lds, gc);
        else sweep_table<8, ST, DEBUG, STAGED>(P, W, I, lds, gc);
    }
}

// Wide path (class 2): product modes with KP up to 16 and any record size,
// 32-bit float offsets, tables in global memory.
template <int KP, typename ST, bool DEBUG>
__device__ void sweep_wide(const SweepParams &P, const Work &W) {
    using Q = Quad<ST>;
    cint32_t *d = W.d;
    const int K = d[0], n_groups = d[10];
    cint32_t *grp = d + d[11];
    const float *tab = P.table + d[3];
    char *states = reinterpret_cast<char *>(P.states);
    const int64_t vstride = node_bytes<ST>(P.m, P.ld);
    const __amdgpu_buffer_rsrc_t own = node_rsrc<ST>(states, W.node, vstride);
    // lanes take (column, replica quad) pairs, consecutive lanes consecutive
    // columns of one quad
    const int64_t c0 = W.q0 * 4;
    const int ncols = (int)((W.q1 * 4 < P.n_cols ? W.q1 * 4 : P.n_cols) - c0);
    const int nrq = (W.r1 - W.r0 + 3) >> 2;
    for (int t = threadIdx.x; t < ncols * nrq; t += kSweepBlock) {
        const int rq = t / ncols;
        const int64_t j = c0 + (t - rq * ncols);
        if (P.obs[(int64_t)W.node * P.ld + j] != 0) continue;
        const int rb = W.r0 + 4 * rq;
        const int nrep = W.r1 - rb < 4 ? W.r1 - rb : 4;
        const uint32_t qoff = quad_boff<ST>(rb >> 2, P.ld, j);
        typename Q::V cur = load_row<ST>(states, W.node, vstride, qoff);
        float w[4][KP];
        wide_product<KP, ST, false>(grp, n_groups, tab, states, vstride, qoff, nrep, w);
        bool low = false;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            float Z = 0.f;
#pragma unroll
            for (int k = 0; k < KP; ++k) Z += w[c][k];
            low |= c < nrep && !(Z >= kUnderflowZ);
        }
        if (low) wide_product<KP, ST, true>(grp, n_groups, tab, states, vstride, qoff, nrep, w);
        const Philox4 rnd = gibbs_block(P, W.node, rb >> 2, j);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            if (c >= nrep) continue;
            if (DEBUG) {
                float Z = 0.f;
#pragma unroll
                for (int k = 0; k < KP; ++k) Z += w[c][k];
                write_probs(P, W.node, rb + c, j, w[c], K, Z);
            }
            running_sums<KP>(w[c]);
            cur = Q::put(cur, c, draw_sums<KP>(w[c], K, uniform24(rnd.w[c])));
        }
        Q::store_buffer(own, qoff, cur);
    }
}

template <typename ST, bool DEBUG>
__global__ __launch_bounds__(kSweepBlock) void sweep_wide_kernel(SweepParams P) {
    if (P.ids) P.sweep_id = P.ids[0];
    const Work W = block_work(P);
    const int KP = W.d[1];
    if (KP == 2) sweep_wide<2, ST, DEBUG>(P, W);
    else if (KP == 4) sweep_wide<4, ST, DEBUG>(P, W);
    else if (KP == 6) sweep_wide<6, ST, DEBUG>(P, W);
    else if (KP == 8) sweep_wide<8, ST, DEBUG>(P, W);
    else sweep_wide<16, ST, DEBUG>(P, W);
}

// ------------------------------------------------- generic path, K_i > 16
//
// The weight of state k is kept as (mantissa in [0.5, 1), exponent) and
// renormalised exactly after every factor, so any K fits in a few registers;
// the three passes (largest exponent, total, search) each recompute the
// products by walking the node's wide list for one column.

template <typename ST>
__device__ float weight_ext(cint32_t *d, const float *__restrict__ tab, const char *__restrict__ base,
                            int64_t vstride, int c, int k, int &e) {
    using Q = Quad<ST>;
    cint32_t *g = d + d[11];
    const int n_groups = d[10];
    float mnt = 1.f;
    e = 0;
    for (int j = 0; j < n_groups; ++j) {
        const int n_e = g[0];
        uint32_t idx = (uint32_t)g[1];
        for (int t = 0; t < n_e; ++t)
            idx += (uint32_t)Q::get(Q::load_at(base + (int64_t)g[2 + 2 * t] * vstride), c) *
                   (uint32_t)g[3 + 2 * t];
        g += 2 + 2 * n_e;
        mnt *= tab[idx + k];
        const int de = __builtin_amdgcn_frexp_expf(mnt);
        mnt = __builtin_ldexpf(mnt, -de);
        e += de;
    }
    return mnt;
}

template <typename ST, bool DEBUG>
__global__ __launch_bounds__(kSweepBlock) void sweep_generic_kernel(SweepParams P) {
    if (P.ids) P.sweep_id = P.ids[0];
    using Q = Quad<ST>;
    const Work W = block_work(P);
    cint32_t *d = W.d;
    const int K = d[0];
    const float *tab = P.table + d[3];
    char *states = reinterpret_cast<char *>(P.states);
    const int64_t vstride = node_bytes<ST>(P.m, P.ld);
    const int64_t c0 = W.q0 * 4;
    const int ncols = (int)((W.q1 * 4 < P.n_cols ? W.q1 * 4 : P.n_cols) - c0);
    const int nrq = (W.r1 - W.r0 + 3) >> 2;
    for (int t = threadIdx.x; t < ncols * nrq; t += kSweepBlock) {
        const int rq = t / ncols;
        const int64_t j = c0 + (t - rq * ncols);
        if (P.obs[(int64_t)W.node * P.ld + j] != 0) continue;
        const int rb = W.r0 + 4 * rq;
        const int nrep = W.r1 - rb < 4 ? W.r1 - rb : 4;
        const int64_t qe = quad_boff<ST>(rb >> 2, P.ld, j);  // the quad's byte offset in a node block
        const char *base = states + qe;
        char *own = states + (int64_t)W.node * vstride + qe;
        typename Q::V cur = Q::load_at(own);
        const Philox4 rnd = gibbs_block(P, W.node, rb >> 2, j);
        for (int c = 0; c < nrep; ++c) {
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
            const float t_u = uniform24(rnd.w[c]) * Z;
            float S = 0.f;
            int pick = -1, last_pos = 0;
            for (int k = 0; k < K; ++k) {
                int e;
                const float wk = __builtin_ldexpf(weight_ext<ST>(d, tab, base, vstride, c, k, e), e - E);
                S += wk;
                if (wk > 0.f) last_pos = k;
                if (pick < 0 && t_u < S) pick = k;
                if (DEBUG && j >= P.win_begin && j < P.win_begin + P.win)
                    P.probs[(((int64_t)W.node * P.m + rb + c) * P.win + (j - P.win_begin)) * P.max_card + k] =
                        wk / Z;
            }
            if (pick < 0) pick = last_pos;
            cur = Q::put(cur, c, pick);
        }
        Q::store_at(own, cur);
    }
}

// ------------------------------------------------------ threshold tables

// One thread per blanket configuration of a table-mode node: decodes the
// configuration (blanket nodes in ascending id, last fastest), forms the log
// conditional in fp64 from max(theta, FLT_MIN), and stores the thresholds
// T_k = ceil(2^24 * S_k / Z) for k < K-1, padded with 2^24.
constexpr int kMaxBlanketTable = 24;

__device__ __forceinline__ void build_thresholds_block(
    int32_t blk, const int32_t *__restrict__ cprog, const int32_t *__restrict__ cprog_off,
    const int32_t *__restrict__ blk_prog, const int32_t *__restrict__ blk_first,
    const float *__restrict__ cpts, uint32_t *__restrict__ cond) {
#pragma clang fp contract(off)
    const int32_t *P = cprog + cprog_off[blk_prog[blk]];
    const int K = P[0], KT = P[1], coff = P[2], ncfg = P[3], nbl = P[4];
    const int cfg = blk_first[blk] + (int)threadIdx.x;
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

__global__ __launch_bounds__(kBlock) void build_thresholds_kernel(
    const int32_t *__restrict__ cprog, const int32_t *__restrict__ cprog_off,
    const int32_t *__restrict__ blk_prog, const int32_t *__restrict__ blk_first,
    const float *__restrict__ cpts, uint32_t *__restrict__ cond) {
    build_thresholds_block((int32_t)blockIdx.x, cprog, cprog_off, blk_prog, blk_first, cpts, cond);
}
// ---------------------------------------------------------------- table build

__device__ __forceinline__ void build_tables_block(
    int32_t blk, const Segment *__restrict__ segs, const int32_t *__restrict__ blk_seg,
    const int32_t *__restrict__ blk_first, const float *__restrict__ cpts, float *__restrict__ table) {
    const Segment sg = segs[blk_seg[blk]];
    const int32_t grp = blk_first[blk] + (int32_t)threadIdx.x;
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

__global__ __launch_bounds__(kBlock) void build_tables_kernel(
    const Segment *__restrict__ segs, const int32_t *__restrict__ blk_seg,
    const int32_t *__restrict__ blk_first, const float *__restrict__ cpts, float *__restrict__ table) {
    build_tables_block((int32_t)blockIdx.x, segs, blk_seg, blk_first, cpts, table);
}

// ---------------------------------------------------------------- counts

__global__ void fill_zero_kernel(int32_t *p, int64_t count) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * blockDim.x)
        p[i] = 0;
}

// What precedes a step's sweep, in one launch: blocks [0, n_build) build the
// k-vector tables, the next n_cond blocks the threshold tables (both from the
// CPTs), and the last n_zero blocks clear the count histogram (grid-stride).
// Each part runs the same code per element as its own kernel; on small
// minibatches a step's launches cost more than their work.
struct PrepareArgs {
    const Segment *segs;
    const int32_t *blk_seg, *blk_first;
    float *table;
    const int32_t *cprog, *cprog_off, *cblk_prog, *cblk_first;
    uint32_t *cond;
    const float *cpts;
    int32_t *zero;
    int64_t zero_count;
    int32_t n_build, n_cond, n_zero;
};

__global__ __launch_bounds__(kBlock) void prepare_step_kernel(PrepareArgs A) {
    const int32_t b = (int32_t)blockIdx.x;
    if (b < A.n_build) {
        build_tables_block(b, A.segs, A.blk_seg, A.blk_first, A.cpts, A.table);
    } else if (b < A.n_build + A.n_cond) {
        build_thresholds_block(b - A.n_build, A.cprog, A.cprog_off, A.cblk_prog, A.cblk_first, A.cpts, A.cond);
    } else {
        const int64_t z = b - A.n_build - A.n_cond;
        for (int64_t i = z * kBlock + threadIdx.x; i < A.zero_count; i += (int64_t)A.n_zero * kBlock)
            A.zero[i] = 0;
    }
}

// Histogram of (parent row, state) for one node over a run of columns and all
// m replicas.  Small CPTs (<= kRepBins bins) use kCopies interleaved LDS
// copies, lane l adding into copy l % kCopies, so lanes hitting the same bin
// rarely collide; larger CPTs share one LDS histogram of at most kLdsBins
// bins: a count work item covers the bins [lo, lo + kLdsBins) of its node,
// and a CPT with more bins has one work item per range, each reading the
// node's rows and counting only its own bins.  CPTs beyond kCountSplitBins
// (lo = -1) go straight to global atomics.  Each block flushes its non-zero
// bins once.
constexpr int kCopies = 32;
constexpr int kRepBins = 256;
constexpr int kLdsBins = kCountLdsBins;
static_assert(kCopies * kRepBins <= kLdsBins, "LDS budget");

// The state quads of NQ adjacent columns of one replica quad at byte offset
// boff.  WIDE (rows of at least NQ columns): one 16-byte load per 16 bytes of
// states (8-byte for two int8 quads); a lane whose columns would run past the
// end of the row (whole false) loads its quads one at a time instead, each
// wholly inside or wholly past the node's buffer.  Not WIDE: always one at a
// time.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <typename ST, int NQ>
struct Span {
    using V = typename Quad<ST>::V;
    static constexpr int kWords = NQ * Quad<ST>::kBytes / 4;  // 32-bit words of NQ quads
    uint32_t w[kWords];                                       // the quads as loaded

    template <bool WIDE>
    __device__ void load(const void *__restrict__ states, int32_t node, int64_t vstride, uint32_t boff,
                         bool whole) {
        const __amdgpu_buffer_rsrc_t r = node_rsrc<ST>(states, node, vstride);
        if (WIDE && whole) {
            if constexpr (kWords == 2) {
                const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)boff, 0, 0);
                w[0] = v.x;
                w[1] = v.y;
            } else {
                static_assert(kWords % 4 == 0, "16-byte pieces");
#pragma unroll
                for (int i = 0; i < kWords / 4; ++i) {
                    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)boff + 16 * i, 0, 0);
                    w[4 * i] = v.x;
                    w[4 * i + 1] = v.y;
                    w[4 * i + 2] = v.z;
                    w[4 * i + 3] = v.w;
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < NQ; ++j) {
                const V q = Quad<ST>::load_buffer(r, boff + (uint32_t)(j * Quad<ST>::kBytes));
                if constexpr (Quad<ST>::kBytes == 2) {
                    if (j & 1) w[j >> 1] |= q << 16;
                    else w[j >> 1] = q;
                } else if constexpr (Quad<ST>::kBytes == 4) {
                    w[j] = q;
                } else {
                    w[2 * j] = q.x;
                    w[2 * j + 1] = q.y;
                }
            }
        }
    }

    // state quad of column j
    __device__ V quad(int j) const {
        if constexpr (Quad<ST>::kBytes == 2) return (w[j >> 1] >> (16 * (j & 1))) & 0xffffu;
        else if constexpr (Quad<ST>::kBytes == 4) return w[j];
        else return make_uint2(w[2 * j], w[2 * j + 1]);
    }

    // The span's NQ x 4 states as 16-bit lanes, 2 NQ words: for 8- and
    // 16-bit states two slots of one column per word (Quad::split); for 4-bit
    // states one slot of two adjacent columns per word (a 32-bit word holds
    // the quads of columns 2p and 2p + 1, so one shift and mask per slot).
    __device__ void lanes(uint32_t (&L)[2 * NQ]) const {
        if constexpr (Quad<ST>::kBytes == 2) {
#pragma unroll
            for (int p = 0; p < NQ / 2; ++p)
#pragma unroll
                for (int c = 0; c < 4; ++c) L[4 * p + c] = (w[p] >> (4 * c)) & 0x000f000fu;
        } else {
#pragma unroll
            for (int h = 0; h < NQ; ++h) {
                uint32_t p2[2];
                Quad<ST>::split(quad(h), p2);
                L[2 * h] = p2[0];
                L[2 * h + 1] = p2[1];
            }
        }
    }

    // the 16-bit lane of (column h, slot c) in the layout of lanes()
    __device__ static uint32_t lane_of(const uint32_t (&L)[2 * NQ], int h, int c) {
        uint32_t v, hi;
        if constexpr (Quad<ST>::kBytes == 2) {
            v = L[4 * (h >> 1) + c];
            hi = h & 1;
        } else {
            v = L[2 * h + Quad<ST>::word_of(c)];
            hi = Quad<ST>::half_of(c);
        }
        return hi ? v >> 16 : v & 0xffffu;
    }
};

constexpr int kCountQuads = 3;  // replica quads whose rows are loaded together (m = 10: all of them)

// Histogram of (parent row, state) for one node over a slab of columns and a
// range of replica quads (block geometry as the sweep's, decode_block).  Bins
// are counted with packed 16-bit arithmetic (two lanes per word, as in the
// sweep) when the node has at most 2^16 bins, else with 32-bit indices.
// Padding slots (replicas >= m) and columns past the slab are not counted.
template <typename ST, bool WIDE>
__global__ __launch_bounds__(kBlock) void count_kernel(const int32_t *__restrict__ cdesc,
                                                      const int32_t *__restrict__ cdesc_off,
                                                      const int32_t *__restrict__ cwork,
                                                      int32_t count, int64_t n_slabs,
                                                      int64_t cols_per_block, int32_t rsplit,
                                                      int32_t quads_per_block,
                                                      const void *__restrict__ states, int32_t m,
                                                      int64_t col0, int64_t n_cols, int64_t ld,
                                                      int32_t *__restrict__ counts) {
    using Q = Quad<ST>;
    __shared__ int32_t hist[kLdsBins];
    uint32_t node_u;
    int64_t slab;
    decode_block(blockIdx.x, (uint32_t)count, node_u, slab);
    if (slab >= n_slabs) return;  // uniform across the block
    const int node = as_const(cwork)[2 * node_u];
    const int lo = as_const(cwork)[2 * node_u + 1];
    cint32_t *d = as_const(cdesc) + as_const(cdesc_off)[node];
    const int K = d[0], n_par = d[1], nbins = d[2], off = d[3];
    cint32_t *par = d + 4;
    // histogram modes: 0 interleaved copies, 1 the whole CPT in one shared
    // histogram, 3 one bin range of a larger CPT in it, 2 global atomics
    const int mode = nbins <= kRepBins ? 0 : (lo < 0 ? 2 : (lo == 0 && nbins <= kLdsBins ? 1 : 3));
    const int range = nbins - lo < kLdsBins ? nbins - lo : kLdsBins;  // modes 1, 3: this item's bins
    const int lds_words = mode == 0 ? nbins * kCopies : (mode == 2 ? 0 : range);
    for (int b = threadIdx.x; b < lds_words; b += kBlock) hist[b] = 0;
    __syncthreads();
    const int copy = threadIdx.x & (kCopies - 1);
    // a slab is a column run and a range [qb, qe) of replica quads; absolute
    // columns of the row: [c0, c1) inside [col0, col0 + n_cols)
    const int rpart = (int)(slab % rsplit);
    slab /= rsplit;
    const int mq = (m + 3) >> 2;
    const int qb = rpart * quads_per_block;
    const int qe = qb + quads_per_block < mq ? qb + quads_per_block : mq;
    const int64_t c0 = col0 + slab * cols_per_block;
    const int64_t c1 = c0 + cols_per_block < col0 + n_cols ? c0 + cols_per_block : col0 + n_cols;
    const int64_t vstride = node_bytes<ST>(m, ld);
    const bool packed = nbins <= 65536;
    // a lane covers NQ adjacent columns (one state quad each), read with wide
    // loads per replica quad
    constexpr int NQ = kCountQuadsPerLane;
    using S = Span<ST, NQ>;
    if (!packed) {
        // 32-bit indices (more than 2^16 bins, global atomics): one replica
        // quad at a time
        for (int64_t col = c0 + NQ * (int64_t)threadIdx.x; col < c1; col += NQ * kBlock) {
            const int nvalid = c1 - col < NQ ? (int)(c1 - col) : NQ;
            const bool whole = col + NQ <= ld;
            for (int rq = qb; rq < qe; ++rq) {
                const int nrep = m - 4 * rq < 4 ? m - 4 * rq : 4;
                const uint32_t boff = quad_boff<ST>(rq, ld, col);
                S own;
                own.template load<WIDE>(states, node, vstride, boff, whole);
                uint32_t u[NQ][4];
#pragma unroll
                for (int h = 0; h < NQ; ++h)
#pragma unroll
                    for (int c = 0; c < 4; ++c) u[h][c] = 0;
                for (int q = 0; q < n_par; ++q) {
                    const uint32_t stride = (uint32_t)par[2 * q + 1];
                    S sp;
                    sp.template load<WIDE>(states, par[2 * q], vstride, boff, whole);
#pragma unroll
                    for (int h = 0; h < NQ; ++h)
#pragma unroll
                        for (int c = 0; c < 4; ++c) u[h][c] += (uint32_t)Q::get(sp.quad(h), c) * stride;
                }
#pragma unroll
                for (int h = 0; h < NQ; ++h)
#pragma unroll
                    for (int c = 0; c < 4; ++c)
                        if (h < nvalid && c < nrep)
                            atomicAdd(&counts[off + u[h][c] * (uint32_t)K + (uint32_t)Q::get(own.quad(h), c)], 1);
            }
        }
        return;
    }
    // packed 16-bit bins.  The histogram mode is uniform per block, so each
    // mode has its own copy of the column loop: no per-slot dispatch.
    auto run = [&](auto md) {
        constexpr int MD = decltype(md)::value;
        auto add = [&](uint32_t bin) {
            if constexpr (MD == 0) {
                atomicAdd(&hist[bin * kCopies + copy], 1);
            } else if constexpr (MD == 1) {
                atomicAdd(&hist[bin], 1);
            } else if constexpr (MD == 3) {
                const uint32_t hb = bin - (uint32_t)lo;
                if (hb < (uint32_t)range) atomicAdd(&hist[hb], 1);
            } else {
                atomicAdd(&counts[off + bin], 1);
            }
        };
        for (int64_t col = c0 + NQ * (int64_t)threadIdx.x; col < c1; col += NQ * kBlock) {
            const int nvalid = c1 - col < NQ ? (int)(c1 - col) : NQ;
            const bool whole = col + NQ <= ld;
            // every lane of the wave holds NQ columns (uniform)
            const bool full = __all(nvalid == NQ);
            for (int rq0 = qb; rq0 < qe; rq0 += kCountQuads) {
                const int nq = qe - rq0 < kCountQuads ? qe - rq0 : kCountQuads;
                uint32_t boff[kCountQuads];
                S own[kCountQuads];
                // every slot loads (a fixed count keeps all loads in flight at
                // once); slots past the last replica quad read through the
                // node's buffer resource past its end, which returns 0 without
                // a memory access, and their values are never used
#pragma unroll
                for (int t = 0; t < kCountQuads; ++t) {
                    boff[t] = quad_boff<ST>(rq0 + t, ld, col);
                    own[t].template load<WIDE>(states, node, vstride, boff[t], whole);
                }
                // bin = sum over parents of x_p * (stride_p * K) + x_node
                uint32_t Pk[kCountQuads][2 * NQ];
#pragma unroll
                for (int t = 0; t < kCountQuads; ++t) own[t].lanes(Pk[t]);
                for (int q = 0; q < n_par; ++q) {
                    const uint32_t mult = (uint32_t)(par[2 * q + 1] * K) * 0x10001u;
                    S sp[kCountQuads];
#pragma unroll
                    for (int t = 0; t < kCountQuads; ++t)
                        sp[t].template load<WIDE>(states, par[2 * q], vstride, boff[t], whole);
                    // slots past the last quad compute on zeros and are never
                    // counted: no exit from the unrolled loop
#pragma unroll
                    for (int t = 0; t < kCountQuads; ++t) {
                        uint32_t L[2 * NQ];
                        sp[t].lanes(L);
#pragma unroll
                        for (int i = 0; i < 2 * NQ; ++i) Pk[t][i] = pk_mad_u16(L[i], mult, Pk[t][i]);
                    }
                }
#pragma unroll
                for (int t = 0; t < kCountQuads; ++t) {
                    if (t >= nq) continue;  // uniform
                    const int nrep = m - 4 * (rq0 + t) < 4 ? m - 4 * (rq0 + t) : 4;
                    if (full) {
                        // uniform branches only
#pragma unroll
                        for (int c = 0; c < 4; ++c)
                            if (c < nrep)
#pragma unroll
                                for (int h = 0; h < NQ; ++h) add(S::lane_of(Pk[t], h, c));
                    } else {
#pragma unroll
                        for (int c = 0; c < 4; ++c)
                            if (c < nrep)
#pragma unroll
                                for (int h = 0; h < NQ; ++h)
                                    if (h < nvalid) add(S::lane_of(Pk[t], h, c));
                    }
                }
            }
        }
    };
    if (mode == 0) run(std::integral_constant<int, 0>{});
    else if (mode == 1) run(std::integral_constant<int, 1>{});
    else if (mode == 3) run(std::integral_constant<int, 3>{});
    else run(std::integral_constant<int, 2>{});
    if (mode == 2) return;
    __syncthreads();
    for (int b = threadIdx.x; b < (mode == 0 ? nbins : range); b += kBlock) {
        int v;
        if (mode == 0) {
            v = 0;
#pragma unroll 8
            for (int k = 0; k < kCopies; ++k) v += hist[b * kCopies + ((k + b) & (kCopies - 1))];
        } else {
            v = hist[b];
        }
        if (v) atomicAdd(&counts[off + lo + b], v);
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

template <typename T>
__global__ void gamma_kernel(const T *__restrict__ totals, double alpha, uint32_t k0, uint32_t k1,
                             uint32_t update_id, const uint32_t *__restrict__ ids, double *__restrict__ g,
                             int64_t total) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= total) return;
    const uint32_t u = ids ? ids[1] : update_id;
    g[e] = gamma_mt(alpha + (double)totals[e], (uint32_t)e, u, k0, k1);
}

// The moving sum of a step's counts and the Gamma draw of every CPT entry
// from the updated total, in one launch: per entry, the arithmetic of
// moving_sum_kernel followed by that of gamma_kernel<int32_t>.
__global__ void moving_sum_gamma_kernel(const int32_t *__restrict__ newc, int32_t *__restrict__ mb,
                                        int32_t *__restrict__ totals, double alpha, uint32_t k0, uint32_t k1,
                                        uint32_t update_id, const uint32_t *__restrict__ ids,
                                        double *__restrict__ g, int64_t total) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= total) return;
    const int32_t nv = newc[e];
    const int32_t delta = nv - mb[e];
    mb[e] = nv;
    const int32_t t = totals[e] + delta;
    totals[e] = t;
    const uint32_t u = ids ? ids[1] : update_id;
    g[e] = gamma_mt(alpha + (double)t, (uint32_t)e, u, k0, k1);
}

// The id pair of a replayed step graph moves on by (d0, d1) after the step.
__global__ void advance_ids_kernel(uint32_t *ids, uint32_t d0, uint32_t d1) {
    if (threadIdx.x == 0) {
        ids[0] += d0;
        ids[1] += d1;
    }
}

// Exponential moving sum of the counts (Sec. 4, for datasets whose
// per-minibatch counts are not kept): totals = decay * totals + new, in fp64
// with the product rounded before the sum.
__global__ void ema_kernel(const int32_t *__restrict__ newc, double *__restrict__ totals, double decay,
                           int64_t total) {
#pragma clang fp contract(off)
    for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x)
        totals[e] = decay * totals[e] + (double)newc[e];
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

// ---------------------------------------------------------------- ingest

// Known entries of one minibatch, CSR with rows = nodes (Sec. 4: a typically
// sparse variables x cases matrix), into the dense layout: one thread per
// stored entry.  Two lanes find the rows of the block's first and last
// entries (the largest i with row_ptr[i] <= e), and each thread searches only
// between them (usually one or two rows).  The entry's value goes to every
// replica (Sec. 4: m copies of the known data) and its obs byte is set; obs was
// cleared by the launcher.  Of repeated (ascending) columns in a row only the
// last entry writes.
__device__ __forceinline__ int row_of(const int64_t *__restrict__ row_ptr, int lo, int hi, int64_t e) {
    while (hi - lo > 1) {  // row_ptr[lo] <= e < row_ptr[hi]
        const int mid = (lo + hi) >> 1;
        if (row_ptr[mid] <= e) lo = mid;
        else hi = mid;
    }
    return lo;
}

template <typename ST>
__global__ __launch_bounds__(kBlock) void expand_kernel(const int64_t *__restrict__ row_ptr, int32_t n,
                                                        const int32_t *__restrict__ col_idx,
                                                        const typename ElemOf<ST>::T *__restrict__ values,
                                                        int64_t nnz, int32_t m, int64_t n_cols, int64_t ld,
                                                        char *__restrict__ states, uint8_t *__restrict__ obs) {
    __shared__ int32_t span[2];
    const int64_t e0 = (int64_t)blockIdx.x * kBlock;
    const int64_t e_last = e0 + kBlock <= nnz ? e0 + kBlock - 1 : nnz - 1;
    if (threadIdx.x < 2) span[threadIdx.x] = row_of(row_ptr, 0, n, threadIdx.x == 0 ? e0 : e_last);
    __syncthreads();
    const int64_t e = e0 + threadIdx.x;
    if (e >= nnz) return;
    const int lo = row_of(row_ptr, span[0], span[1] + 1, e);
    const int64_t j = col_idx[e];
    if (j < 0 || j >= n_cols) return;
    if (e + 1 < row_ptr[lo + 1] && col_idx[e + 1] == j) return;  // a later entry of this column
    obs[(int64_t)lo * ld + j] = 1;
    // every slot of the column's state quads, padding included, takes the value
    const typename Quad<ST>::V v = Quad<ST>::splat((int)values[e]);
    char *dst = states + (int64_t)lo * node_bytes<ST>(m, ld) + quad_boff<ST>(0, ld, j);
    const int mq = (m + 3) >> 2;
    for (int rq = 0; rq < mq; ++rq) Quad<ST>::store_at(dst + (int64_t)rq * ld * Quad<ST>::kBytes, v);
}

// Random initial latent states (Sec. 5.2): one thread per (node, column
// quad), looping over the replicas; for replica r the Philox block at counter
// {g >> 2, i, r | 2 << 24, 0} (g the global column of the quad's first
// column) gives word c to column c, and the state is ((w >> 8) * K_i) >> 24 =
// floor(U * K_i) exactly.  The quad's obs dword is read once; for each
// replica quad, the state quads of the four columns are read, the latent
// columns' real slots replaced, and written back.  Observed entries and
// padding slots keep their values.
template <typename ST>
__global__ __launch_bounds__(kBlock) void init_latent_kernel(const int32_t *__restrict__ cdesc,
                                                             const int32_t *__restrict__ cdesc_off,
                                                             int32_t n, int32_t m, int64_t n_cols,
                                                             int64_t ld, int64_t col_offset, uint32_t k0,
                                                             uint32_t k1, char *__restrict__ states,
                                                             const uint8_t *__restrict__ obs) {
    using Q = Quad<ST>;
    const int64_t quads = (n_cols + 3) >> 2;
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)n * quads) return;
    const int64_t q = t % quads;
    const int i = (int)(t / quads);
    const int64_t col = 4 * q;
    const uint32_t ob = *reinterpret_cast<const uint32_t *>(obs + (int64_t)i * ld + col);
    int lat = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c)
        if (((ob >> (8 * c)) & 0xffu) == 0 && col + c < n_cols) lat |= 1 << c;
    if (!lat) return;
    const uint32_t K = (uint32_t)cdesc[cdesc_off[i]];
    const int mq = (m + 3) >> 2;
    for (int rq = 0; rq < mq; ++rq) {
        char *p = states + (int64_t)i * node_bytes<ST>(m, ld) + quad_boff<ST>(rq, ld, col);
        typename Q::V v[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) v[c] = Q::load_at(p + c * Q::kBytes);
        for (int s = 0; s < 4 && 4 * rq + s < m; ++s) {
            const Philox4 b = philox4x32_10((uint32_t)((col_offset >> 2) + q), (uint32_t)i,
                                            (uint32_t)(4 * rq + s) | (2u << 24), 0u, k0, k1);
#pragma unroll
            for (int c = 0; c < 4; ++c)
                if ((lat >> c) & 1) v[c] = Q::put(v[c], s, (int)(((uint64_t)(b.w[c] >> 8) * K) >> 24));
        }
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if ((lat >> c) & 1) Q::store_at(p + c * Q::kBytes, v[c]);
    }
}

// ---------------------------------------------------------------- prediction

// Held-out prediction (Sec. 6): with the CPTs frozen, hits[i][j] counts the
// replicas whose state equals the test entry's true value target[i][j] (-1:
// not a test entry).  One thread per (node, column quad): the quad's targets
// and hit counters are read once, the replicas' state quads are compared in
// turn, and the counters are written back.
template <typename ST>
__global__ __launch_bounds__(kBlock) void hits_kernel(const char *__restrict__ states,
                                                      const typename ElemOf<ST>::T *__restrict__ target,
                                                      int32_t n, int32_t m, int64_t n_cols, int64_t ld,
                                                      int32_t *__restrict__ hits) {
    using Q = Quad<ST>;
    using E = typename ElemOf<ST>::T;
    using QE = Quad<E>;  // four adjacent targets
    const int64_t quads = (n_cols + 3) >> 2;
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)n * quads) return;
    const int64_t q = t % quads;
    const int i = (int)(t / quads);
    const int64_t col = 4 * q;
    const typename QE::V tg = QE::load(target + (int64_t)i * ld + col);
    int want[4], any = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        want[c] = (int)(E)QE::get(tg, c);
        if (col + c >= n_cols) want[c] = -1;
        any |= want[c] >= 0;
    }
    if (!any) return;
    int add[4] = {0, 0, 0, 0};
    const int mq = (m + 3) >> 2;
    for (int rq = 0; rq < mq; ++rq) {
        const char *p = states + (int64_t)i * node_bytes<ST>(m, ld) + quad_boff<ST>(rq, ld, col);
        const int nrep = m - 4 * rq < 4 ? m - 4 * rq : 4;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const typename Q::V v = Q::load_at(p + c * Q::kBytes);  // column col + c, four replica slots
            for (int sl = 0; sl < nrep; ++sl)
                add[c] += (uint32_t)Q::get(v, sl) == ((uint32_t)want[c] & Q::kMask) ? 1 : 0;
        }
    }
    int4 *h = reinterpret_cast<int4 *>(hits + (int64_t)i * ld + col);
    int4 cur = *h;
    if (want[0] >= 0) cur.x += add[0];
    if (want[1] >= 0) cur.y += add[1];
    if (want[2] >= 0) cur.z += add[2];
    if (want[3] >= 0) cur.w += add[3];
    *h = cur;
}

// ------------------------------------------------------ compact host state
//
// Out-of-core passes that keep only the latent entries on the host (the
// known data stay on the device): per minibatch, the latent states of node i
// are stored compactly, replica r's at [node_off[i] + r * L_i, + L_i), in
// ascending column order (L_i = the node's latent columns in the minibatch).
// node_off holds the offsets of the whole host array; off0 is the first of
// the minibatch, where the device buffer starts.  A block of these kernels
// takes one node and one chunk of kCompactChunk columns; a lane reads the obs
// word of its 4 columns.

constexpr int kCompactChunk = 4 * kBlock;

// Latent columns of each (node, chunk) of the minibatch [c0, c0 + cols).
__global__ __launch_bounds__(kBlock) void compact_counts_kernel(const uint8_t *__restrict__ obs, int64_t obs_ld,
                                                                int64_t c0, int64_t cols, int32_t chunks,
                                                                int32_t *__restrict__ counts) {
    __shared__ int32_t total;
    const int node = (int)(blockIdx.x / chunks), chunk = (int)(blockIdx.x % chunks);
    if (threadIdx.x == 0) total = 0;
    __syncthreads();
    const int64_t j = (int64_t)chunk * kCompactChunk + 4 * threadIdx.x;
    int cnt = 0;
    if (j < cols) {
        const uint32_t ob = *reinterpret_cast<const uint32_t *>(obs + (int64_t)node * obs_ld + c0 + j);
#pragma unroll
        for (int c = 0; c < 4; ++c) cnt += (((ob >> (8 * c)) & 0xffu) == 0 && j + c < cols) ? 1 : 0;
    }
    if (cnt) atomicAdd(&total, cnt);
    __syncthreads();
    if (threadIdx.x == 0) counts[blockIdx.x] = total;
}

// Latent columns of each node in the minibatch [c0, c0 + cols): one block per
// node walks the columns.
__global__ __launch_bounds__(kBlock) void compact_node_counts_kernel(const uint8_t *__restrict__ obs, int64_t obs_ld,
                                                                     int64_t c0, int64_t cols,
                                                                     int32_t *__restrict__ counts) {
    __shared__ int32_t total;
    const int node = blockIdx.x;
    if (threadIdx.x == 0) total = 0;
    __syncthreads();
    int cnt = 0;
    for (int64_t j = 4 * (int64_t)threadIdx.x; j < cols; j += kCompactChunk) {
        const uint32_t ob = *reinterpret_cast<const uint32_t *>(obs + (int64_t)node * obs_ld + c0 + j);
#pragma unroll
        for (int c = 0; c < 4; ++c) cnt += (((ob >> (8 * c)) & 0xffu) == 0 && j + c < cols) ? 1 : 0;
    }
    if (cnt) atomicAdd(&total, cnt);
    __syncthreads();
    if (threadIdx.x == 0) counts[node] = total;
}

// Per node, the counts of its chunks become their exclusive prefix sums.
__global__ __launch_bounds__(kBlock) void compact_prefix_kernel(int32_t *__restrict__ counts, int32_t n,
                                                                int32_t chunks) {
    const int node = blockIdx.x * kBlock + threadIdx.x;
    if (node >= n) return;
    int32_t *c = counts + (int64_t)node * chunks, run = 0;
    for (int k = 0; k < chunks; ++k) {
        const int32_t v = c[k];
        c[k] = run;
        run += v;
    }
}

// Rank, among the node's latent columns of the minibatch, of the first latent
// column of each lane's quad (block-wide prefix sum over the lanes' obs words),
// and the lane's latent mask.
__device__ __forceinline__ int compact_rank(const uint8_t *__restrict__ obs, int64_t obs_ld, int64_t c0,
                                            int64_t cols, int node, int chunk, const int32_t *__restrict__ prefix,
                                            int32_t chunks, int32_t *wave_n, int &lat) {
    const int64_t j = (int64_t)chunk * kCompactChunk + 4 * threadIdx.x;
    lat = 0;
    if (j < cols) {
        const uint32_t ob = *reinterpret_cast<const uint32_t *>(obs + (int64_t)node * obs_ld + c0 + j);
#pragma unroll
        for (int c = 0; c < 4; ++c)
            if (((ob >> (8 * c)) & 0xffu) == 0 && j + c < cols) lat |= 1 << c;
    }
    const int cnt = __builtin_popcount(lat);
    const uint64_t b0 = __ballot(cnt & 1), b1 = __ballot(cnt & 2), b2 = __ballot(cnt & 4);
    auto below = [](uint64_t b) {
        return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(b >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)b, 0u));
    };
    const int pre = below(b0) + 2 * below(b1) + 4 * below(b2);
    const int wave = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0)
        wave_n[wave] = __builtin_popcountll(b0) + 2 * __builtin_popcountll(b1) + 4 * __builtin_popcountll(b2);
    __syncthreads();
    int base = prefix[(int64_t)node * chunks + chunk];
#pragma unroll
    for (int v = 0; v < kBlock / 64; ++v) base += v < wave ? wave_n[v] : 0;
    return base + pre;
}

// Dense slot of a minibatch from the device-resident known data and the
// compact latent states: every replica takes the known value at an observed
// column and its compact latent state at a latent one (padding slots: the
// known value, or 0 at a latent column); the slot's obs rows are copied as
// well.  Columns [cols, slot_ld) are left untouched.
template <typename ST>
__global__ __launch_bounds__(kBlock) void expand_compact_kernel(
    const uint8_t *__restrict__ obs, const typename ElemOf<ST>::T *__restrict__ data, int64_t obs_ld, int64_t c0,
    int64_t cols,
    int32_t m, int32_t chunks, const int32_t *__restrict__ prefix, const int64_t *__restrict__ node_off,
    int64_t off0, const typename ElemOf<ST>::T *__restrict__ lat_states, char *__restrict__ states,
    uint8_t *__restrict__ obs_slot,
    int64_t slot_ld) {
    using Q = Quad<ST>;
    using E = typename ElemOf<ST>::T;
    using QE = Quad<E>;
    __shared__ int32_t wave_n[kBlock / 64];
    const int node = (int)(blockIdx.x / chunks), chunk = (int)(blockIdx.x % chunks);
    int lat;
    const int rank = compact_rank(obs, obs_ld, c0, cols, node, chunk, prefix, chunks, wave_n, lat);
    const int64_t j = (int64_t)chunk * kCompactChunk + 4 * threadIdx.x;
    if (j >= cols) return;
    const int64_t L = (node_off[node + 1] - node_off[node]) / m;
    const E *lat_node = lat_states + (node_off[node] - off0);
    *reinterpret_cast<uint32_t *>(obs_slot + (int64_t)node * slot_ld + j) =
        *reinterpret_cast<const uint32_t *>(obs + (int64_t)node * obs_ld + c0 + j);
    const typename QE::V known = QE::load(data + (int64_t)node * obs_ld + c0 + j);  // columns j .. j + 3
    int kc[4];  // compact rank of each latent column of the lane
    {
        int k = rank;
#pragma unroll
        for (int c = 0; c < 4; ++c) kc[c] = ((lat >> c) & 1) ? k++ : -1;
    }
    const int mq = (m + 3) >> 2;
    char *dst = states + (int64_t)node * node_bytes<ST>(m, slot_ld) + quad_boff<ST>(0, slot_ld, j);
    for (int rq = 0; rq < mq; ++rq) {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            typename Q::V v = Q::splat(kc[c] >= 0 ? 0 : QE::get(known, c));
            if (kc[c] >= 0)
                for (int sl = 0; sl < 4 && 4 * rq + sl < m; ++sl)
                    v = Q::put(v, sl, (int)lat_node[(int64_t)(4 * rq + sl) * L + kc[c]]);
            Q::store_at(dst + ((int64_t)rq * slot_ld + c) * Q::kBytes, v);
        }
    }
}

// The inverse: the latent states of the dense slot back into compact form.
template <typename ST>
__global__ __launch_bounds__(kBlock) void gather_compact_kernel(
    const uint8_t *__restrict__ obs, int64_t obs_ld, int64_t c0, int64_t cols, int32_t m, int32_t chunks,
    const int32_t *__restrict__ prefix, const int64_t *__restrict__ node_off, int64_t off0,
    const char *__restrict__ states, int64_t slot_ld, typename ElemOf<ST>::T *__restrict__ lat_states) {
    using Q = Quad<ST>;
    __shared__ int32_t wave_n[kBlock / 64];
    const int node = (int)(blockIdx.x / chunks), chunk = (int)(blockIdx.x % chunks);
    int lat;
    const int rank = compact_rank(obs, obs_ld, c0, cols, node, chunk, prefix, chunks, wave_n, lat);
    const int64_t j = (int64_t)chunk * kCompactChunk + 4 * threadIdx.x;
    if (j >= cols || !lat) return;
    const int64_t L = (node_off[node + 1] - node_off[node]) / m;
    typename ElemOf<ST>::T *lat_node = lat_states + (node_off[node] - off0);
    const int mq = (m + 3) >> 2;
    const char *src = states + (int64_t)node * node_bytes<ST>(m, slot_ld) + quad_boff<ST>(0, slot_ld, j);
    int k = rank;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        if (!((lat >> c) & 1)) continue;
        for (int rq = 0; rq < mq; ++rq) {
            const typename Q::V v = Q::load_at(src + ((int64_t)rq * slot_ld + c) * Q::kBytes);
            for (int sl = 0; sl < 4 && 4 * rq + sl < m; ++sl)
                lat_node[(int64_t)(4 * rq + sl) * L + k] = (typename ElemOf<ST>::T)Q::get(v, sl);
        }
        ++k;
    }
}

// ---------------------------------------------------------------- annealing

// SAME annealing (Sec. 3: raising the replication factor during sampling):
// dst (m2 replicas) takes replica r < m of src (m replicas) and, for r >= m, a
// copy of replica r mod m; padding slots of dst take the same rule.  One
// thread per (node, column): the source quads of the column are read once and
// the destination quads assembled slot by slot.
template <typename ST>
__global__ __launch_bounds__(kBlock) void grow_kernel(const char *__restrict__ src, int32_t m, char *__restrict__ dst,
                                                      int32_t m2, int32_t n, int64_t ld) {
    using Q = Quad<ST>;
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (int64_t)n * ld) return;
    const int i = (int)(t / ld);
    const int64_t j = t - (int64_t)i * ld;
    const char *s = src + (int64_t)i * node_bytes<ST>(m, ld) + quad_boff<ST>(0, ld, j);
    char *d = dst + (int64_t)i * node_bytes<ST>(m2, ld) + quad_boff<ST>(0, ld, j);
    const int mq2 = (m2 + 3) >> 2;
    for (int rq = 0; rq < mq2; ++rq) {
        typename Q::V v{};
#pragma unroll
        for (int sl = 0; sl < 4; ++sl) {
            const int r = (4 * rq + sl) % m;
            v = Q::put(v, sl, Q::get(Q::load_at(s + (int64_t)(r >> 2) * ld * Q::kBytes), r & 3));
        }
        Q::store_at(d + (int64_t)rq * ld * Q::kBytes, v);
    }
}

}  // namespace dev

// ================================================================= launchers

namespace {
inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

// Calls f with a value of the state type of a format: 4-bit (Nib), 8- or
// 16-bit states.
template <typename F>
void by_format(int32_t bits, F &&f) {
    if (bits == 4) f(dev::Nib{});
    else if (bits == 8) f(int8_t{});
    else f(int16_t{});
}

// Count histogram of the allocation-free count entry point: a file-scope
// device array (each device holds its own copy until the process ends).  In
// host code `scratch` names a host-side stand-in, not device memory; its
// device address comes from hipGetSymbolAddress, resolved once per device.
static __device__ __align__(256) int32_t scratch[kScratchCountEntries];

std::mutex g_scratch_mu;
std::vector<int32_t *> g_scratch_ptr;  // indexed by device ordinal
}  // namespace

hipError_t scratch_counts(int device, int32_t **out) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (device < 0) return hipErrorInvalidDevice;
    if ((int)g_scratch_ptr.size() <= device) g_scratch_ptr.resize(device + 1, nullptr);
    if (!g_scratch_ptr[device]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        g_scratch_ptr[device] = static_cast<int32_t *>(p);
    }
    *out = g_scratch_ptr[device];
    return hipSuccess;
}

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
    const dim3 blk(dev::kSweepBlock);
    if (klass == 0) {
        if (dbg) hipLaunchKernelGGL((dev::sweep_fast_kernel<ST, true, true>), grid, blk, lds_bytes, stream, P);
        else hipLaunchKernelGGL((dev::sweep_fast_kernel<ST, false, true>), grid, blk, lds_bytes, stream, P);
    } else if (klass == 1 && lds_bytes > 0) {
        // partially staged records
        if (dbg) hipLaunchKernelGGL((dev::sweep_fast_kernel<ST, true, true>), grid, blk, lds_bytes, stream, P);
        else hipLaunchKernelGGL((dev::sweep_fast_kernel<ST, false, true>), grid, blk, lds_bytes, stream, P);
    } else if (klass == 1) {
        if (dbg) hipLaunchKernelGGL((dev::sweep_fast_kernel<ST, true, false>), grid, blk, 0, stream, P);
        else hipLaunchKernelGGL((dev::sweep_fast_kernel<ST, false, false>), grid, blk, 0, stream, P);
    } else if (klass == 2) {
        if (dbg) hipLaunchKernelGGL((dev::sweep_wide_kernel<ST, true>), grid, blk, 0, stream, P);
        else hipLaunchKernelGGL((dev::sweep_wide_kernel<ST, false>), grid, blk, 0, stream, P);
    } else {
        if (dbg) hipLaunchKernelGGL((dev::sweep_generic_kernel<ST, true>), grid, blk, 0, stream, P);
        else hipLaunchKernelGGL((dev::sweep_generic_kernel<ST, false>), grid, blk, 0, stream, P);
    }
}

}  // namespace

hipError_t launch_sweep(SweepParams P, int32_t begin, int32_t count, int32_t klass,
                        int32_t lds_bytes, int32_t state_bits, hipStream_t stream) {
    if (count <= 0 || P.n_cols <= 0) return hipSuccess;
    // Slabs of kSweepQuadsPerLane column quads per lane.  A block that stages
    // its node's table in LDS (class 0) takes all replicas, so that the copy
    // is paid once per column chunk, and replicas are split only when that
    // leaves fewer than kMinSweepBlocks blocks; the other classes take one
    // replica quad per block: smaller slabs keep the blanket rows and the
    // global tables that the resident blocks gather from in L2 (measured
    // faster).  A block's replica range is always whole state quads (the
    // last one ends at m), so that no two blocks write one quad.
    const int64_t quads = (P.n_cols + 3) / 4;
    P.quads_per_block = (int64_t)dev::kSweepBlock * dev::kSweepQuadsPerLane;
    // the fast kernel draws replicas in quads (one Philox block each), so a
    // block's replica range is whole quads except at the end
    const int64_t m_quads = (P.m + 3) / 4;
    // small launches (few nodes or columns) take narrower column chunks, down
    // to 256 columns, so that even with one replica quad per block they fill
    // the device with blocks
    if (klass <= 1)
        while (P.quads_per_block > dev::kMinSweepQuads &&
               count * ((quads + P.quads_per_block - 1) / P.quads_per_block) * m_quads < dev::kMinSweepBlocks)
            P.quads_per_block /= 2;
    const int64_t chunks = (quads + P.quads_per_block - 1) / P.quads_per_block;
    int64_t rsplit = klass == 0 ? (dev::kMinSweepBlocks + count * chunks - 1) / (count * chunks) : m_quads;
    if (rsplit > m_quads) rsplit = m_quads;
    if (rsplit < 1) rsplit = 1;
    const int64_t quads_per_block = (m_quads + rsplit - 1) / rsplit;
    P.rsplit = (int32_t)((m_quads + quads_per_block - 1) / quads_per_block);
    P.reps_per_block = (int32_t)(4 * quads_per_block);
    P.n_slabs = chunks * P.rsplit;
    P.count = count;
    P.begin = begin;
    const int64_t rounds = (P.n_slabs + dev::kXcds - 1) / dev::kXcds;
    const int64_t blocks = rounds * dev::kXcds * count;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    const dim3 grid((unsigned)blocks);
    by_format(state_bits, [&](auto tag) { sweep_class<decltype(tag)>(P, klass, lds_bytes, grid, stream); });
    return hipGetLastError();
}

hipError_t launch_build_thresholds(const DeviceTables &t, const float *cpts, uint32_t *cond,
                                   hipStream_t stream) {
    if (t.n_cond_blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(dev::build_thresholds_kernel, dim3(t.n_cond_blocks), dim3(dev::kBlock), 0,
                       stream, t.cprog, t.cprog_off, t.cblk_prog, t.cblk_first, cpts, cond);
    return hipGetLastError();
}

hipError_t launch_prepare(const DeviceTables &t, const float *cpts, float *table, uint32_t *cond, int32_t *zero,
                          int64_t zero_count, hipStream_t stream) {
    dev::PrepareArgs A;
    A.segs = t.segs;
    A.blk_seg = t.blk_seg;
    A.blk_first = t.blk_first;
    A.table = table;
    A.cprog = t.cprog;
    A.cprog_off = t.cprog_off;
    A.cblk_prog = t.cblk_prog;
    A.cblk_first = t.cblk_first;
    A.cond = cond;
    A.cpts = cpts;
    A.zero = zero;
    A.zero_count = zero_count > 0 ? zero_count : 0;
    A.n_build = t.n_build_blocks;
    A.n_cond = t.n_cond_blocks;
    int64_t nz = A.zero_count > 0 ? (int64_t)blocks_for(A.zero_count, dev::kBlock) : 0;
    if (nz > 1024) nz = 1024;
    A.n_zero = (int32_t)nz;
    const int64_t blocks = (int64_t)A.n_build + A.n_cond + A.n_zero;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(dev::prepare_step_kernel, dim3((unsigned)blocks), dim3(dev::kBlock), 0, stream, A);
    return hipGetLastError();
}

hipError_t launch_moving_sum_gamma(const int32_t *newc, int32_t *mb, int32_t *totals, double alpha, uint32_t key0,
                                   uint32_t key1, uint32_t update_id, const uint32_t *ids, double *g, int64_t total,
                                   hipStream_t stream) {
    if (total <= 0) return hipSuccess;
    hipLaunchKernelGGL(dev::moving_sum_gamma_kernel, dim3(blocks_for(total, dev::kBlock)), dim3(dev::kBlock), 0,
                       stream, newc, mb, totals, alpha, key0, key1, update_id, ids, g, total);
    return hipGetLastError();
}

hipError_t launch_fill_zero(int32_t *p, int64_t count, hipStream_t stream) {
    if (count <= 0) return hipSuccess;
    unsigned nb = blocks_for(count, dev::kBlock);
    if (nb > 4096) nb = 4096;
    hipLaunchKernelGGL(dev::fill_zero_kernel, dim3(nb), dim3(dev::kBlock), 0, stream, p, count);
    return hipGetLastError();
}

hipError_t launch_counts(const DeviceTables &t, const void *states, int32_t state_bits,
                         int32_t m, int64_t col0, int64_t n_cols, int64_t ld, int32_t *counts,
                         hipStream_t stream) {
    if (n_cols <= 0) return hipSuccess;
    const int32_t n = t.n_cwork;
    // one node x 4096 columns (two lane iterations of kCountQuadsPerLane
    // columns) x all replica quads per block, XCD-swizzled like the sweep;
    // launches with few blocks take one lane iteration (2048 columns) per
    // block
    const int64_t mq = (m + 3) / 4;
    const int64_t quad_runs = (mq + dev::kCountQuads - 1) / dev::kCountQuads;
    int64_t cols_per_block = 2 * dev::kBlock * dev::kCountQuadsPerLane;
    if ((int64_t)n * ((n_cols + cols_per_block - 1) / cols_per_block) * quad_runs < dev::kMinSweepBlocks)
        cols_per_block /= 2;
    const int64_t col_slabs = (n_cols + cols_per_block - 1) / cols_per_block;
    // small launches split the replica quads (in runs of kCountQuads) over
    // blocks until there are kMinSweepBlocks blocks, so that they fill the
    // device
    int64_t rparts = (dev::kMinSweepBlocks + (int64_t)n * col_slabs - 1) / ((int64_t)n * col_slabs);
    if (rparts > quad_runs) rparts = quad_runs;
    if (rparts < 1) rparts = 1;
    const int32_t quads_per_block = (int32_t)(dev::kCountQuads * ((quad_runs + rparts - 1) / rparts));
    const int32_t rsplit = (int32_t)((mq + quads_per_block - 1) / quads_per_block);
    const int64_t n_slabs = col_slabs * rsplit;
    const int64_t rounds = (n_slabs + dev::kXcds - 1) / dev::kXcds;
    const int64_t blocks = rounds * dev::kXcds * n;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    const dim3 grid((unsigned)blocks);
#define SAME_LAUNCH_COUNTS(ST, WIDE)                                                                    \
    hipLaunchKernelGGL((dev::count_kernel<ST, WIDE>), grid, dim3(dev::kBlock), 0, stream, t.cdesc, t.cdesc_off, \
                       t.cwork, n, n_slabs, cols_per_block, rsplit, quads_per_block, states, m, col0, \
                       n_cols, ld, counts)
    // rows of at least kCountQuadsPerLane columns take the wide loads
    by_format(state_bits, [&](auto tag) {
        using ST = decltype(tag);
        if (ld >= dev::kCountQuadsPerLane) SAME_LAUNCH_COUNTS(ST, true);
        else SAME_LAUNCH_COUNTS(ST, false);
    });
#undef SAME_LAUNCH_COUNTS
    return hipGetLastError();
}

hipError_t launch_expand(const int64_t *row_ptr, int32_t n, const int32_t *col_idx, const void *values,
                         int64_t nnz, int32_t m, int64_t n_cols, int64_t ld, int32_t state_bits,
                         void *states, uint8_t *obs, hipStream_t stream) {
    // obs [n][ld] bytes (ld a multiple of 4) cleared as words, then the entries
    hipError_t e = launch_fill_zero(reinterpret_cast<int32_t *>(obs), (int64_t)n * ld / 4, stream);
    if (e != hipSuccess || nnz <= 0) return e;
    const int64_t blocks = (nnz + dev::kBlock - 1) / dev::kBlock;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    by_format(state_bits, [&](auto tag) {
        using ST = decltype(tag);
        using E = typename dev::ElemOf<ST>::T;
        hipLaunchKernelGGL(dev::expand_kernel<ST>, dim3((unsigned)blocks), dim3(dev::kBlock), 0, stream, row_ptr, n,
                           col_idx, (const E *)values, nnz, m, n_cols, ld, (char *)states, obs);
    });
    return hipGetLastError();
}

hipError_t launch_init_latent(const DeviceTables &t, int32_t n, int32_t m, int64_t n_cols, int64_t ld,
                              int64_t col_offset, uint32_t key0, uint32_t key1, int32_t state_bits,
                              void *states, const uint8_t *obs, hipStream_t stream) {
    const int64_t items = (int64_t)n * ((n_cols + 3) / 4);
    if (items <= 0) return hipSuccess;
    const int64_t blocks = (items + dev::kBlock - 1) / dev::kBlock;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    by_format(state_bits, [&](auto tag) {
        hipLaunchKernelGGL(dev::init_latent_kernel<decltype(tag)>, dim3((unsigned)blocks), dim3(dev::kBlock), 0,
                           stream, t.cdesc, t.cdesc_off, n, m, n_cols, ld, col_offset, key0, key1, (char *)states,
                           obs);
    });
    return hipGetLastError();
}

hipError_t launch_hits(const void *states, const void *target, int32_t n, int32_t m, int64_t n_cols, int64_t ld,
                       int32_t state_bits, int32_t *hits, hipStream_t stream) {
    const int64_t items = (int64_t)n * ((n_cols + 3) / 4);
    if (items <= 0) return hipSuccess;
    const int64_t blocks = (items + dev::kBlock - 1) / dev::kBlock;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    by_format(state_bits, [&](auto tag) {
        using ST = decltype(tag);
        using E = typename dev::ElemOf<ST>::T;
        hipLaunchKernelGGL(dev::hits_kernel<ST>, dim3((unsigned)blocks), dim3(dev::kBlock), 0, stream,
                           (const char *)states, (const E *)target, n, m, n_cols, ld, hits);
    });
    return hipGetLastError();
}

hipError_t launch_compact_node_counts(const uint8_t *obs, int64_t obs_ld, int64_t c0, int64_t cols, int32_t n,
                                      int32_t *counts, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(dev::compact_node_counts_kernel, dim3((unsigned)n), dim3(dev::kBlock), 0, stream, obs, obs_ld,
                       c0, cols, counts);
    return hipGetLastError();
}

hipError_t launch_compact_counts(const uint8_t *obs, int64_t obs_ld, int64_t c0, int64_t cols, int32_t n,
                                 int32_t *counts, bool prefix, hipStream_t stream) {
    const int32_t chunks = (int32_t)((cols + dev::kCompactChunk - 1) / dev::kCompactChunk);
    if (cols <= 0 || n <= 0) return hipSuccess;
    hipLaunchKernelGGL(dev::compact_counts_kernel, dim3((unsigned)((int64_t)n * chunks)), dim3(dev::kBlock), 0,
                       stream, obs, obs_ld, c0, cols, chunks, counts);
    if (prefix)
        hipLaunchKernelGGL(dev::compact_prefix_kernel, dim3(blocks_for(n, dev::kBlock)), dim3(dev::kBlock), 0,
                           stream, counts, n, chunks);
    return hipGetLastError();
}

hipError_t launch_expand_compact(const uint8_t *obs, const void *data, int64_t obs_ld, int64_t c0, int64_t cols,
                                 int32_t n, int32_t m, const int32_t *prefix, const int64_t *node_off, int64_t off0,
                                 const void *lat_states, void *states, uint8_t *obs_slot, int64_t slot_ld,
                                 int32_t state_bits, hipStream_t stream) {
    const int32_t chunks = (int32_t)((cols + dev::kCompactChunk - 1) / dev::kCompactChunk);
    if (cols <= 0 || n <= 0) return hipSuccess;
    const dim3 grid((unsigned)((int64_t)n * chunks));
    by_format(state_bits, [&](auto tag) {
        using ST = decltype(tag);
        using E = typename dev::ElemOf<ST>::T;
        hipLaunchKernelGGL(dev::expand_compact_kernel<ST>, grid, dim3(dev::kBlock), 0, stream, obs, (const E *)data,
                           obs_ld, c0, cols, m, chunks, prefix, node_off, off0, (const E *)lat_states,
                           (char *)states, obs_slot, slot_ld);
    });
    return hipGetLastError();
}

hipError_t launch_gather_compact(const uint8_t *obs, int64_t obs_ld, int64_t c0, int64_t cols, int32_t n, int32_t m,
                                 const int32_t *prefix, const int64_t *node_off, int64_t off0, const void *states,
                                 int64_t slot_ld, void *lat_states, int32_t state_bits, hipStream_t stream) {
    const int32_t chunks = (int32_t)((cols + dev::kCompactChunk - 1) / dev::kCompactChunk);
    if (cols <= 0 || n <= 0) return hipSuccess;
    const dim3 grid((unsigned)((int64_t)n * chunks));
    by_format(state_bits, [&](auto tag) {
        using ST = decltype(tag);
        using E = typename dev::ElemOf<ST>::T;
        hipLaunchKernelGGL(dev::gather_compact_kernel<ST>, grid, dim3(dev::kBlock), 0, stream, obs, obs_ld, c0, cols,
                           m, chunks, prefix, node_off, off0, (const char *)states, slot_ld, (E *)lat_states);
    });
    return hipGetLastError();
}

hipError_t launch_grow(const void *src, int32_t m, void *dst, int32_t m2, int32_t n, int64_t ld,
                       int32_t state_bits, hipStream_t stream) {
    const int64_t items = (int64_t)n * ld;
    if (items <= 0) return hipSuccess;
    const int64_t blocks = (items + dev::kBlock - 1) / dev::kBlock;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    by_format(state_bits, [&](auto tag) {
        hipLaunchKernelGGL(dev::grow_kernel<decltype(tag)>, dim3((unsigned)blocks), dim3(dev::kBlock), 0, stream,
                           (const char *)src, m, (char *)dst, m2, n, ld);
    });
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

template <typename T>
hipError_t launch_gamma_t(const T *totals, double alpha, uint32_t key0, uint32_t key1, uint32_t update_id,
                          const uint32_t *ids, double *g, int64_t total, hipStream_t stream) {
    if (total <= 0) return hipSuccess;
    hipLaunchKernelGGL(dev::gamma_kernel<T>, dim3(blocks_for(total, dev::kBlock)), dim3(dev::kBlock), 0, stream,
                       totals, alpha, key0, key1, update_id, ids, g, total);
    return hipGetLastError();
}

hipError_t launch_gamma(const int32_t *totals, double alpha, uint32_t key0, uint32_t key1,
                        uint32_t update_id, const uint32_t *ids, double *g, int64_t total,
                        hipStream_t stream) {
    return launch_gamma_t(totals, alpha, key0, key1, update_id, ids, g, total, stream);
}

hipError_t launch_gamma(const double *totals, double alpha, uint32_t key0, uint32_t key1,
                        uint32_t update_id, const uint32_t *ids, double *g, int64_t total,
                        hipStream_t stream) {
    return launch_gamma_t(totals, alpha, key0, key1, update_id, ids, g, total, stream);
}

hipError_t launch_advance_ids(uint32_t *ids, uint32_t d0, uint32_t d1, hipStream_t stream) {
    hipLaunchKernelGGL(dev::advance_ids_kernel, dim3(1), dim3(64), 0, stream, ids, d0, d1);
    return hipGetLastError();
}

hipError_t launch_ema(const int32_t *newc, double *totals, double decay, int64_t total, hipStream_t stream) {
    if (total <= 0) return hipSuccess;
    unsigned nb = blocks_for(total, dev::kBlock);
    if (nb > 4096) nb = 4096;
    hipLaunchKernelGGL(dev::ema_kernel, dim3(nb), dim3(dev::kBlock), 0, stream, newc, totals, decay, total);
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
