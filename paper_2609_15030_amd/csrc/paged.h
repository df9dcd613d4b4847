// Paged fp32 state pool: scatter (save) and gather (restore) of whole pages.
// One workgroup moves one page with 16-byte lanes, several loads in flight
// per lane, non-temporal stores (the copy is read once and not reused by the
// copying kernel).
#pragma once
#include "la_common.h"

namespace la {

constexpr int kPageThreads = 256;
constexpr int kPageUnroll = 4;

__device__ inline void copy_page(const f32x4 *__restrict__ src, f32x4 *__restrict__ dst,
                                 int64_t nvec) {
    int64_t v = threadIdx.x;
    const int64_t step = kPageThreads * kPageUnroll;
    for (; v + (kPageUnroll - 1) * kPageThreads < nvec; v += step) {
        f32x4 x[kPageUnroll];
#pragma unroll
        for (int u = 0; u < kPageUnroll; ++u) x[u] = __builtin_nontemporal_load(src + v + u * kPageThreads);
#pragma unroll
        for (int u = 0; u < kPageUnroll; ++u) __builtin_nontemporal_store(x[u], dst + v + u * kPageThreads);
    }
    for (; v < nvec; v += kPageThreads) __builtin_nontemporal_store(__builtin_nontemporal_load(src + v), dst + v);
}

__global__ __launch_bounds__(kPageThreads) void page_save_kernel(const f32x4 *states, int64_t nvec,
                                                                 f32x4 *pool, int64_t n_pages,
                                                                 const int32_t *ids, int32_t *err) {
    const int64_t item = blockIdx.x;
    const int32_t pid = ids[item];
    if (pid == -1) return;
    if (pid < 0 || pid >= n_pages) {
        if (threadIdx.x == 0 && err) atomicAdd(err, 1);
        return;
    }
    copy_page(states + item * nvec, pool + (int64_t)pid * nvec, nvec);
}

__global__ __launch_bounds__(kPageThreads) void page_restore_kernel(const f32x4 *pool, int64_t n_pages,
                                                                    const int32_t *ids, f32x4 *states,
                                                                    int64_t nvec, int32_t *err) {
    const int64_t item = blockIdx.x;
    const int32_t pid = ids[item];
    f32x4 *dst = states + item * nvec;
    if (pid == -1) {
        for (int64_t v = threadIdx.x; v < nvec; v += kPageThreads)
            __builtin_nontemporal_store(zero4(), dst + v);
        return;
    }
    if (pid < 0 || pid >= n_pages) {
        if (threadIdx.x == 0 && err) atomicAdd(err, 1);
        return;
    }
    copy_page(pool + (int64_t)pid * nvec, dst, nvec);
}

}  // namespace la
