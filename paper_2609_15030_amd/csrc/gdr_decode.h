// Decode continuation: one token per sequence through the gated delta rule,
// from and back into the fp32 state in HBM (the recurrent state of section
// 2.1, advanced one generated token at a time after a cold prefill or a
// reload; sections 5.1 and 5.4 compare such continuations).
//
// Per (sequence, head), with alpha = exp(g):
//   pred = S^T k                 (literal)   or  alpha S^T k  (decayed delta)
//   u    = beta (v - pred)
//   S    = alpha S + k u^T
//   o    = scale S^T q
// Columns of S are independent, so a workgroup owns 32 of them: 256 threads,
// thread (rg, cg) holds rows [rg R, rg R + R) x columns [4 cg, 4 cg + 4) of
// its column block (R = DK / 32), reads them once (16-byte loads, 128 bytes
// per row per 8 threads), and writes them back once.  The two dk reductions
// (pred and o) go through LDS.  fp32 arithmetic; the step moves 2 * 4 dk dv
// bytes of state per head and is HBM-bound.
#pragma once
#include "la_common.h"

namespace la {

struct DecodeArgs {
    const void *q, *k, *v;        // [n_seqs, H, dk | dv] io type
    const float *g, *beta;        // [n_seqs, H]
    float *state;                 // [n_seqs, H, DK, DV], updated in place
    void *o;                      // [n_seqs, H, DV] io type
    int32_t n_seqs, n_heads, variant;
    float scale;
};

constexpr int kDecodeThreads = 256;
constexpr int kDecodeCols = 32;   // state columns per workgroup

template <typename T, int DK, int DV>
__global__ __launch_bounds__(kDecodeThreads) void gdr_decode_kernel(DecodeArgs a) {
    constexpr int CB = DV / kDecodeCols;    // column blocks per head
    constexpr int RG = kDecodeThreads / (kDecodeCols / 4);   // row groups (32)
    constexpr int R = DK / RG;              // rows per thread
    static_assert(R >= 1 && R * RG == DK, "rows");
    __shared__ float kq[2][DK];
    __shared__ float4 red[RG][kDecodeCols / 4];

    const int tid = threadIdx.x, cg = tid & 7, rg = tid >> 3;
    const int unit = blockIdx.x / CB, cb = blockIdx.x % CB;
    if (unit >= a.n_seqs * a.n_heads) return;
    const int col = cb * kDecodeCols + 4 * cg;
    const T *qv = (const T *)a.q + (size_t)unit * DK;
    const T *kv = (const T *)a.k + (size_t)unit * DK;
    float *S = a.state + (size_t)unit * DK * DV;

    // the state rows this thread owns, in flight first
    float4 s[R];
#pragma unroll
    for (int r = 0; r < R; ++r) s[r] = *(const float4 *)&S[(size_t)(rg * R + r) * DV + col];
    for (int i = tid; i < DK; i += kDecodeThreads) {
        kq[0][i] = to_f32(kv[i]);
        kq[1][i] = to_f32(qv[i]);
    }
    const float alpha = expf(a.g[unit]), beta = a.beta[unit];
    float4 vv;
    {
        const T *vp = (const T *)a.v + (size_t)unit * DV + col;
        vv = make_float4(to_f32(vp[0]), to_f32(vp[1]), to_f32(vp[2]), to_f32(vp[3]));
    }
    __syncthreads();

    // pred = S^T k over this thread's rows, then across the row groups
    float4 p = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const float kr = kq[0][rg * R + r];
        p.x += s[r].x * kr;
        p.y += s[r].y * kr;
        p.z += s[r].z * kr;
        p.w += s[r].w * kr;
    }
    red[rg][cg] = p;
    __syncthreads();
    float4 pred = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int i = 0; i < RG; ++i) {
        const float4 x = red[i][cg];
        pred.x += x.x;
        pred.y += x.y;
        pred.z += x.z;
        pred.w += x.w;
    }
    const float pa = a.variant == 0 ? 1.f : alpha;
    const float4 u = make_float4(beta * (vv.x - pa * pred.x), beta * (vv.y - pa * pred.y),
                                 beta * (vv.z - pa * pred.z), beta * (vv.w - pa * pred.w));
    // S = alpha S + k u^T, written back; o = S^T q over this thread's rows
    float4 oo = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const float kr = kq[0][rg * R + r], qr = kq[1][rg * R + r];
        float4 x = s[r];
        x.x = alpha * x.x + kr * u.x;
        x.y = alpha * x.y + kr * u.y;
        x.z = alpha * x.z + kr * u.z;
        x.w = alpha * x.w + kr * u.w;
        *(float4 *)&S[(size_t)(rg * R + r) * DV + col] = x;
        oo.x += x.x * qr;
        oo.y += x.y * qr;
        oo.z += x.z * qr;
        oo.w += x.w * qr;
    }
    __syncthreads();   // every thread is done reading pred's partials
    red[rg][cg] = oo;
    __syncthreads();
    if (rg == 0) {
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int i = 0; i < RG; ++i) {
            const float4 x = red[i][cg];
            acc.x += x.x;
            acc.y += x.y;
            acc.z += x.z;
            acc.w += x.w;
        }
        T *op = (T *)a.o + (size_t)unit * DV + col;
        op[0] = from_f32<T>(acc.x * a.scale);
        op[1] = from_f32<T>(acc.y * a.scale);
        op[2] = from_f32<T>(acc.z * a.scale);
        op[3] = from_f32<T>(acc.w * a.scale);
    }
}

}  // namespace la
