// Output read-out of a chunk, one 16-column tile of the state at a time.
//
// For chunk rows r (tokens) and s, with S_0 the state entering the chunk, U
// the chunk's corrections (U = U~ - W S_0) and
//   P_rs = (q_r . k_s) exp(G_r - G_s) for s <= r, zero above the diagonal
// (written by the preparation kernel), the read-out of the post-update
// state S_r^T q_r is
//   o_r = scale * ( exp(G_r) S_0^T q_r + sum_s P_rs u_s ).
// Per 16-token tile it is computed transposed,
//   O^T = scale * ( (S_0^T Q^T) diag(exp G) + U^T P^T ),
// because then the state and U enter as A operands straight from the scan's
// registers (per lane, the A operand of X^T holds the same values as the B
// operand of X, including the contraction-index permutation perm_row), Q^T
// and P^T are B operands (both written by the preparation kernel in that
// order, read here with whole 16-byte vectors), and each lane ends with 4
// consecutive output columns of one token: one 8-byte (bf16) or 16-byte
// (fp32) store.
//
// The scan kernel's output wave and the split output kernel run this same
// code on the same operands, so both paths produce identical bits.
#pragma once
#include "la_common.h"

namespace la {

constexpr float kLog2eOut = 1.4426950408889634f;

// One chunk's read-out operands that every column tile shares, as one lane
// holds them (g = lane / 16, c = lane % 16):
//   q[mt][f] = Q[16 mt + c][perm_row(f, g)]      (B operand of Q^T, dk permuted)
//   p[mt][f] = P[16 mt + c][perm_row(f, g)]      (B operand of P^T, chunk rows permuted)
//   eg[mt]   = exp(G_{16 mt + c})
template <typename T, int DK> struct OutFrag {
    static constexpr int FS = DK / 4, FU = kChunk / 4;
    T q[4][FS];
    T p[4][FU];
    float eg[4];
};

template <typename T> __device__ inline void buf_store_4(__amdgpu_buffer_rsrc_t r, uint32_t voff, const T *src);
template <> __device__ inline void buf_store_4<__bf16>(__amdgpu_buffer_rsrc_t r, uint32_t voff, const __bf16 *src) {
    buf_store8(*(const uint2 *)src, r, voff, 0u);
}
template <> __device__ inline void buf_store_4<float>(__amdgpu_buffer_rsrc_t r, uint32_t voff, const float *src) {
    buf_store16(*(const uint4 *)src, r, voff, 0u);
}

// Byte range of rows [0, n) of one head in a [tokens, H, D] tensor, counted
// from row 0 of that head: row n and later fall outside it, so buffer
// accesses to them read zero and drop stores (the chunk's ragged tail).
// The value is wave-uniform; readfirstlane keeps it in a scalar register
// (a buffer resource held in vector registers costs a loop per access).
template <typename T> __device__ inline uint32_t head_rows_bytes(int n, int H, int D) {
    const uint32_t b = ((uint32_t)(n - 1) * (uint32_t)H * (uint32_t)D + (uint32_t)D) * (uint32_t)sizeof(T);
    return (uint32_t)__builtin_amdgcn_readfirstlane((int)b);
}

// Issues the loads of one chunk's read-out operands: the Q and P fragments
// and the gates of workspace slot-head sh.
template <typename T, int DK>
__device__ inline void load_out_frag(OutFrag<T, DK> &f, const Workspace &ws, int64_t sh) {
    constexpr int VEC = Vec<T>::N, VS = OutFrag<T, DK>::FS / VEC, VU = OutFrag<T, DK>::FU / VEC;
    const int lane = threadIdx.x & 63, c16 = lane & 15;
    constexpr size_t QE = (size_t)kChunk * DK;       // Q elements per slot-head
    const auto rq = make_rsrc((const T *)ws.qf + sh * QE, QE * sizeof(T));
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int v = 0; v < VS; ++v)
            *(uint4 *)&f.q[mt][v * VEC] = buf_load16(rq, 16u * (uint32_t)lane + 1024u * (mt * VS + v), 0u);
    constexpr size_t PE = (size_t)kChunk * kChunk;   // P elements per slot-head
    const auto rp = make_rsrc((const T *)ws.p + sh * PE, PE * sizeof(T));
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int v = 0; v < VU; ++v)
            *(uint4 *)&f.p[mt][v * VEC] = buf_load16(rp, 16u * (uint32_t)lane + 1024u * (mt * VU + v), 0u);
    // the gates of rows c, 16 + c, 32 + c, 48 + c sit together (G layout)
    const uint4 e = buf_load16(make_rsrc(ws.g + sh * kChunk, kChunk * sizeof(float)), 16u * (uint32_t)c16, 0u);
    f.eg[0] = __uint_as_float(e.x);
    f.eg[1] = __uint_as_float(e.y);
    f.eg[2] = __uint_as_float(e.z);
    f.eg[3] = __uint_as_float(e.w);
}

// O^T for one 16-column tile of the state: sb and ub are the scan's operand
// forms of S_0 (B-operand order of S_0, i.e. A-operand order of S_0^T) and
// of U; o is the output of head h at chunk row 0, rows n and later masked.
template <typename T, int DK>
__device__ inline void out_tile(const OutFrag<T, DK> &f, const T *sb, const T *ub, float scale, T *o, int n,
                                int H, int DV, int tile) {
    using M = MT<T>;
    constexpr int KW = M::KW, FS = OutFrag<T, DK>::FS, FU = OutFrag<T, DK>::FU;
    const int lane = threadIdx.x & 63, g16 = lane >> 4, c16 = lane & 15;
    const auto ro = make_rsrc(o, head_rows_bytes<T>(n, H, DV));
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
        f32x4 acc = zero4();
#pragma unroll
        for (int ks = 0; ks < FS / KW; ++ks) acc = M::mma(M::pack(&sb[ks * KW]), M::pack(&f.q[mt][ks * KW]), acc);
        const float eg = __builtin_amdgcn_exp2f(f.eg[mt] * kLog2eOut);
        acc = acc * eg;
#pragma unroll
        for (int ks = 0; ks < FU / KW; ++ks) acc = M::mma(M::pack(&ub[ks * KW]), M::pack(&f.p[mt][ks * KW]), acc);
        T out[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) out[i] = from_f32<T>(acc[i] * scale);
        const uint32_t voff = ((uint32_t)(16 * mt + c16) * (uint32_t)(H * DV) + (uint32_t)(16 * tile + 4 * g16)) *
                              (uint32_t)sizeof(T);
        buf_store_4<T>(ro, voff, out);
    }
}

struct OutArgs {
    void *o;
    const int32_t *cu;
    int32_t n_seqs, n_heads, C, cps, max_chunks;
    float scale;
    Workspace ws;
    int32_t chunk_major;   // block map (see unit_of_block)
};

// Split output kernel (used when the scan ran without its output wave: the
// two-level scan, the dk-split scan, and a call that runs the output stage
// on its own): one workgroup per (chunk, head, sequence), one wave per
// column tile, reading the state entering the chunk and U from the
// workspace.
template <typename T, int DK, int DV>
__global__ __launch_bounds__(4 * DV) void gdr_out_kernel(OutArgs a) {
    using L = WsLayout<T, DK, DV>;
    constexpr int VEC = Vec<T>::N, FS = DK / 4, FU = kChunk / 4;
    constexpr int VS = FS / VEC, VU = FU / VEC;
    const int lane = threadIdx.x & 63, tile = threadIdx.x >> 6;
    int64_t j;
    int seq, h;
    if (!unit_of_block(a.n_seqs, a.n_heads, a.max_chunks, a.chunk_major != 0, &seq, &h, &j)) return;
    const int H = a.n_heads;
    const int64_t cu0 = a.cu[seq];
    const int len = a.cu[seq + 1] - a.cu[seq];
    if (j >= n_chunks32(len, a.C, a.cps)) return;
    int lo, hi;
    chunk_range32((int)j, len, a.C, a.cps, &lo, &hi);
    const int n = hi - lo;
    const int64_t t0 = cu0 + lo;
    const int64_t sh = (slot_base_dev(cu0, seq, a.C, a.cps) + j) * H + h;

    T sb[FS], ub[FU];
    const auto rs = make_rsrc((const T *)a.ws.sc + sh * L::sc_elems, L::sc_elems * sizeof(T));
    const auto ru = make_rsrc((const T *)a.ws.u + sh * L::u_elems, L::u_elems * sizeof(T));
#pragma unroll
    for (int v = 0; v < VS; ++v) *(uint4 *)&sb[v * VEC] = buf_load16(rs, 16u * lane, 1024u * (tile * VS + v));
#pragma unroll
    for (int v = 0; v < VU; ++v) *(uint4 *)&ub[v * VEC] = buf_load16(ru, 16u * lane, 1024u * (tile * VU + v));
    OutFrag<T, DK> f;
    load_out_frag<T, DK>(f, a.ws, sh);
    out_tile<T, DK>(f, sb, ub, a.scale, (T *)a.o + (t0 * H + h) * DV, n, H, DV, tile);
}

}  // namespace la
