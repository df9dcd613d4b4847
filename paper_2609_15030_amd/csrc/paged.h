// Paged fp32 state pool: scatter (save) and gather (restore) of whole pages.
// One 1,024-lane workgroup moves one page (a 64 KiB page in one pass of four
// 16-byte loads per lane).  Loads are non-temporal (the source is read once);
// stores are ordinary.  On the full 4,096-page pool, saved and restored in
// turn under a random permutation, this was the fastest of the load/store
// cache-policy and shape combinations tried (save 5.5 TB/s, restore
// 6.5 TB/s; non-temporal stores 5.2 / 5.5 TB/s).
#pragma once
#include "la_common.h"

namespace la {

constexpr int kPageThreads = 1024;
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
        for (int u = 0; u < kPageUnroll; ++u) dst[v + u * kPageThreads] = x[u];
    }
    for (; v < nvec; v += kPageThreads) dst[v] = __builtin_nontemporal_load(src + v);
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
        for (int64_t v = threadIdx.x; v < nvec; v += kPageThreads) dst[v] = zero4();
        return;
    }
    if (pid < 0 || pid >= n_pages) {
        if (threadIdx.x == 0 && err) atomicAdd(err, 1);
        return;
    }
    copy_page(pool + (int64_t)pid * nvec, dst, nvec);
}

}  // namespace la
