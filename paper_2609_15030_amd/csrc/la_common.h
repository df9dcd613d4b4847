// Device helpers shared by the gfx950 kernels: MFMA traits, fragment
// layouts, and the chunk plan (which tokens form which chunk, where a
// chunk's intermediates live in the workspace).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace la {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kChunk = 64;        // rows of one chunk tile (the prefill's chunk size)
constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// MFMA traits.  One 16x16 output tile per instruction, fp32 accumulation.
//   bf16: v_mfma_f32_16x16x32_bf16, 8 operand values per lane and k-step.
//   fp32: v_mfma_f32_16x16x4_f32,   1 operand value per lane and k-step.
// Lane layout (lane l, g = l / 16):
//   A (16 x KSTEP): row l % 16, k = g * KW + j   (j < KW)
//   B (KSTEP x 16): col l % 16, k = g * KW + j
//   C (16 x 16):    col l % 16, rows 4 * g + i   (i < 4)
// ---------------------------------------------------------------------------
template <typename T> struct MT;

template <> struct MT<__bf16> {
    static constexpr int KW = 8;
    static constexpr int KSTEP = 32;
    typedef bf16x8 frag;
    __device__ static inline f32x4 mma(frag a, frag b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
    // 8 consecutive values; v must be 16-byte aligned.
    __device__ static inline frag pack(const __bf16 *v) { return *(const frag *)v; }
    // Two runs of 4 consecutive values (8-byte aligned each).
    __device__ static inline frag pack2(const __bf16 *lo, const __bf16 *hi) {
        typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
        const bf16x4 a = *(const bf16x4 *)lo, b = *(const bf16x4 *)hi;
        return frag{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    }
};

template <> struct MT<float> {
    static constexpr int KW = 1;
    static constexpr int KSTEP = 4;
    typedef float frag;
    __device__ static inline f32x4 mma(frag a, frag b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    __device__ static inline frag pack(const float *v) { return v[0]; }
    __device__ static inline frag pack2(const float *lo, const float *) { return lo[0]; }
};

// Raw buffer access: a scalar resource (base, size) plus a per-lane byte
// offset.  Loop-invariant lane offsets keep operand prefetches free of
// per-iteration VGPR address arithmetic; out-of-range reads return zero.
typedef int i32x4 __attribute__((ext_vector_type(4)));
constexpr int kBufferFlags = 0x00020000;   // raw (untyped) dword access

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, (int)bytes, kBufferFlags);
}

__device__ inline uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    const i32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
    return make_uint4((uint32_t)v[0], (uint32_t)v[1], (uint32_t)v[2], (uint32_t)v[3]);
}

// 16 bytes as two 8-byte buffer stores.  A buffer store of more than 8
// bytes reads its data registers after issue: an instruction right behind
// it that rewrites them corrupts the stored words, and the compiler does not
// separate the two when the store's offset sits in a scalar register (the
// form every store here takes).  Stores of 8 bytes or less are free of that
// hazard.  The empty asm statement between the halves keeps the compiler
// from merging them back into one 16-byte store.
__device__ inline void buf_store16(uint4 x, __amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    typedef int i32x2 __attribute__((ext_vector_type(2)));
    const i32x2 lo = {(int)x.x, (int)x.y}, hi = {(int)x.z, (int)x.w};
    __builtin_amdgcn_raw_buffer_store_b64(lo, r, (int)voff, (int)soff, 0);
    __asm__ volatile("" ::: "memory");
    __builtin_amdgcn_raw_buffer_store_b64(hi, r, (int)(voff + 8u), (int)soff, 0);
}

__device__ inline uint2 buf_load8(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    typedef int i32x2 __attribute__((ext_vector_type(2)));
    const i32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)voff, (int)soff, 0);
    return make_uint2((uint32_t)v[0], (uint32_t)v[1]);
}

__device__ inline void buf_store8(uint2 x, __amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    typedef int i32x2 __attribute__((ext_vector_type(2)));
    const i32x2 v = {(int)x.x, (int)x.y};
    __builtin_amdgcn_raw_buffer_store_b64(v, r, (int)voff, (int)soff, 0);
}

__device__ inline float buf_load4f(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)soff, 0));
}

template <typename T> __device__ inline T from_f32(float x);
template <> __device__ inline float from_f32<float>(float x) { return x; }
template <> __device__ inline __bf16 from_f32<__bf16>(float x) { return (__bf16)x; }  // RNE

template <typename T> __device__ inline float to_f32(T x) { return (float)x; }

// Elements of T per 16-byte vector.
template <typename T> struct Vec { static constexpr int N = 16 / sizeof(T); };

__device__ inline f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// Contraction-index permutation.  When the B operand of a product is taken
// straight from a C-layout accumulator (rows 4g+i of each 16-row tile held
// by lane group g), the lane's flat operand index f (f = ks*KW + j over all
// k-steps) stands for accumulator row perm_row(f, g).  The A operand of the
// same product is then loaded at those rows, so no cross-lane shuffle of the
// accumulator is needed.  Every row of the tile set is hit exactly once per
// k-step group, and each k-step covers KSTEP distinct rows.
__device__ __host__ inline int perm_row(int f, int g) {
    return 16 * (f >> 2) + 4 * g + (f & 3);
}

// ---------------------------------------------------------------------------
// Chunk plan.  A sequence's call covers local positions [0, len) starting at
// an absolute position that is a multiple of C.  Chunks never straddle a
// checkpoint position: each C-token segment is cut into ceil(C / 64) chunks
// of at most 64 tokens, so every checkpoint falls on a chunk end.  With C a
// multiple of 64 this is the plain 64-token grid.
// ---------------------------------------------------------------------------
__device__ __host__ inline int chunks_per_interval(int C) { return (C + kChunk - 1) / kChunk; }

__device__ __host__ inline int64_t n_chunks(int64_t len, int64_t C, int cps) {
    const int64_t full = len / C, rem = len % C;
    return full * cps + (rem + kChunk - 1) / kChunk;
}

// Local token range [a, b) of chunk j.
__device__ __host__ inline void chunk_range(int64_t j, int64_t len, int64_t C, int cps,
                                            int64_t *a, int64_t *b) {
    const int64_t seg = j / cps, sub = j % cps;
    const int64_t lo = seg * C + (int64_t)sub * kChunk;
    int64_t hi = lo + kChunk;
    if (hi > (seg + 1) * C) hi = (seg + 1) * C;
    if (hi > len) hi = len;
    *a = lo;
    *b = hi;
}

// 32-bit forms for device code (sequence lengths and C are below 2^31; the
// host validates that), which avoid 64-bit integer division.
__device__ inline int n_chunks32(int len, int C, int cps) {
    const int full = len / C, rem = len - full * C;
    return full * cps + (rem + kChunk - 1) / kChunk;
}

__device__ inline void chunk_range32(int j, int len, int C, int cps, int *a, int *b) {
    const int seg = j / cps, sub = j - seg * cps;
    const int lo = seg * C + sub * kChunk;
    int hi = lo + kChunk;
    if (hi > (seg + 1) * C) hi = (seg + 1) * C;
    if (hi > len) hi = len;
    *a = lo;
    *b = hi;
}

// First workspace slot of sequence i.  A sequence of n tokens has at most
// ceil(n * cps / C) chunks, so slot bases floor((cu[i] * cps + (C - 1) * i) / C)
// give every sequence room for its chunks without a prefix sum over the
// batch: the difference of consecutive bases is at least ceil(n_i * cps / C).
__device__ __host__ inline int64_t slot_base(int64_t cu_i, int64_t i, int64_t C, int cps) {
    return (cu_i * cps + (C - 1) * i) / C;
}

// Device form of slot_base: while the numerator fits 32 bits (every call
// below 2^32 tokens-times-chunks) a 32-bit division replaces the 64-bit one.
__device__ inline int64_t slot_base_dev(int64_t cu_i, int64_t i, int64_t C, int cps) {
    const uint64_t num = (uint64_t)cu_i * (uint64_t)cps + (uint64_t)(C - 1) * (uint64_t)i;
    if (num < (1ull << 32) && C < (1ll << 32)) return (int64_t)((uint32_t)num / (uint32_t)C);
    return (int64_t)(num / (uint64_t)C);
}

__device__ __host__ inline int64_t total_slots(int64_t total_tokens, int64_t n_seqs, int64_t C,
                                               int cps) {
    return slot_base(total_tokens, n_seqs, C, cps);
}

// ---------------------------------------------------------------------------
// XCD-aware block mapping of the per-chunk kernels.  Workgroups are dealt to
// the 8 XCDs round-robin by linear id; each XCD has its own L2.  Two maps:
//   pair-major: (sequence, head) pair p goes to XCD p % 8, as in the scan
//     kernels, so a chain's chunks are prepared where it is scanned;
//     block id = 8 * (chunk + max_chunks * (p / 8)) + p % 8;
//   chunk-major: the units of chunk c of a sequence, for every head, go to
//     XCD c % 8, so the chunk's gates and betas (stored [token, head]: a
//     cache line holds a few tokens of every head) are fetched once into one
//     L2 rather than once per head into several; block id =
//     8 * ((seq * CG + c / 8) * H + head) + c % 8, CG = ceil(max_chunks / 8).
// The host takes chunk-major for launches of many units, where the gathers'
// traffic counts, and pair-major otherwise.
// ---------------------------------------------------------------------------
constexpr int64_t kChunkMajorUnits = 2048;

__host__ inline bool chunk_major_map(int n_seqs, int n_heads, int64_t max_chunks) {
    return (int64_t)n_seqs * n_heads * max_chunks > kChunkMajorUnits;
}

__device__ inline bool unit_of_block(int n_seqs, int n_heads, int max_chunks, bool chunk_major, int *seq,
                                     int *head, int64_t *chunk) {
    // 32-bit arithmetic: a 64-bit division costs hundreds of cycles at the
    // start of every workgroup (grids stay below 2^32)
    const uint32_t b = blockIdx.x;
    const uint32_t x = b & 7, m = b >> 3;
    const uint32_t H = (uint32_t)n_heads;
    uint32_t sq, hd, c;
    if (chunk_major) {
        const uint32_t CG = ((uint32_t)max_chunks + 7) / 8;
        const uint32_t t = m / H;
        hd = m - t * H;
        sq = t / CG;
        c = 8 * (t - sq * CG) + x;
        if (sq >= (uint32_t)n_seqs || c >= (uint32_t)max_chunks) return false;
    } else {
        const uint32_t q = m / (uint32_t)max_chunks;
        const uint32_t pair = x + 8 * q;
        if (pair >= (uint32_t)n_seqs * H) return false;
        c = m - q * (uint32_t)max_chunks;
        sq = pair / H;
        hd = pair - sq * H;
    }
    *seq = (int)sq;
    *head = (int)hd;
    *chunk = (int64_t)c;
    return true;
}

__host__ inline int64_t chunk_grid_blocks(int n_seqs, int n_heads, int64_t max_chunks) {
    if (chunk_major_map(n_seqs, n_heads, max_chunks)) return 8 * ((max_chunks + 7) / 8) * (int64_t)n_seqs * n_heads;
    return 8 * max_chunks * (((int64_t)n_seqs * n_heads + 7) / 8);
}

// ---------------------------------------------------------------------------
// Workspace regions (per slot and head), all produced and consumed on the
// device within one prefill call.
//   W   : -W in A-operand order for the state contraction      [4][DK/4] x 64 lanes, io type
//   KT  : decayed keys^T in A-operand order (chunk rows perm.) [DK/16][16] x 64 lanes, io type
//   UT  : U~ = T diag(beta) V, C-layout per 16x16 tile        [DV/16][4] x 64 lanes x 4, io type
//   G   : chunk-local cumulative gate, row 16 m + c at 4 c + m [64], fp32
//         (a lane's four output rows in one 16-byte load; row 63 stays at 63)
//   SC  : state entering the chunk, B-operand order            [DV/16][DK/4] x 64 lanes, io type
//   U   : U = U~ - W S, B-operand order                        [DV/16][16] x 64 lanes, io type
//   P   : decayed causal Q K^T, per token tile the B operand of P^T (chunk
//         rows permuted like KT)                              [4][16] x 64 lanes, io type
//   QF  : queries, per token tile the B operand of Q^T (dk permuted like W)
//                                                              [4][DK/4] x 64 lanes, io type
// ---------------------------------------------------------------------------
struct Workspace {
    void *w, *kt, *sc, *u, *p, *qf, *ut;
    float *g;
    uint4 *misc;       // fused path: per slot-head, the X fragments and the gate block
};

// U~ tile vector `vec` (= column tile * 4 + row tile) of one slot-head, as
// lane `lane` holds it in the C layout (rows 4 (lane / 16) + i, column
// lane % 16): four consecutive elements of the io type, widened to fp32 as
// the accumulator of U = U~ - W S.
template <typename T>
__device__ inline f32x4 load_ut(__amdgpu_buffer_rsrc_t r, uint32_t lane, uint32_t vec) {
    if constexpr (sizeof(T) == 4) {
        const uint4 x = buf_load16(r, 16u * lane, 1024u * vec);
        return f32x4{__uint_as_float(x.x), __uint_as_float(x.y), __uint_as_float(x.z), __uint_as_float(x.w)};
    } else {
        const uint2 x = buf_load8(r, 8u * lane, 512u * vec);
        return f32x4{__uint_as_float(x.x << 16), __uint_as_float(x.x & 0xffff0000u), __uint_as_float(x.y << 16),
                     __uint_as_float(x.y & 0xffff0000u)};
    }
}

template <typename T, int DK, int DV> struct WsLayout {
    static constexpr size_t w_elems = (size_t)kChunk * DK;      // per slot-head
    static constexpr size_t kt_elems = (size_t)DK * kChunk;
    static constexpr size_t ut_elems = (size_t)kChunk * DV;
    static constexpr size_t g_elems = kChunk;
    static constexpr size_t sc_elems = (size_t)DK * DV;
    static constexpr size_t u_elems = (size_t)kChunk * DV;
    static constexpr size_t p_elems = (size_t)kChunk * kChunk;
    static constexpr size_t qf_elems = (size_t)kChunk * DK;
};

}  // namespace la
