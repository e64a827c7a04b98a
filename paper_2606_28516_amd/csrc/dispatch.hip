// Expert dispatch of the CLEAR-MoE layer: per-tile histogram, exclusive scan
// and a stable counting-sort permutation, plus the inverse-permute combines.
//
// Grouped backend (Sec. III "Dispatch Backends"): tokens are sorted by expert
// into contiguous sub-batches; Algorithm 3 sorts z by the assignment and finds
// the sub-batch boundaries.  Here the boundaries come from a histogram + scan
// that never leaves the device, and the sort is a stable counting sort: the
// assignments a = t*k + j of expert e appear in ascending a.
//
// Tiles are the routing tiles (256 tokens = 256*k assignments).  Inside a tile
// the rank of an assignment among earlier assignments of the same expert is
// found 256 assignments at a time: one ballot per expert per wave gives the
// rank inside the wave (popcount of the lanes below), per-wave totals in LDS
// give the rank across waves, and a running per-expert count carries it over
// the tile's chunks.  Tile bases come from the scan, so no atomics are used
// and the result is deterministic.
#include "kernels.h"

namespace clearmoe {

constexpr int kWaves = kRouteTile / 64;

// Rank of this thread's assignment among equal experts of the chunk.
// Writes per-wave totals to s_wc[w][e].  Returns the rank inside the wave.
__device__ __forceinline__ int wave_rank(bool ok, int ex, int E, int lane, int w,
                                         int (*s_wc)[64]) {
    int rank = 0;
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int e = 0; e < E; ++e) {
        const bool mine = ok && ex == e;
        const uint64_t m = __ballot(mine);
        if (mine) rank = __popcll(m & below);
        if (lane == 0) s_wc[w][e] = __popcll(m);
    }
    return rank;
}

__global__ __launch_bounds__(kRouteTile) void k_tile_hist(const int32_t* __restrict__ idx,
                                                          int64_t T, int E, int k,
                                                          int32_t* __restrict__ tile_counts) {
    __shared__ int s_wc[kWaves][64];
    __shared__ int s_run[64];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t A = T * k;
    const int64_t a0 = static_cast<int64_t>(blockIdx.x) * kRouteTile * k;
    const int64_t na64 = A - a0 < static_cast<int64_t>(kRouteTile) * k ? A - a0
                                                                         : static_cast<int64_t>(kRouteTile) * k;
    const int na = static_cast<int>(na64);
    if (tid < E) s_run[tid] = 0;
    __syncthreads();
    for (int c = 0; c < k; ++c) {
        const int al = c * kRouteTile + tid;
        const int ex = al < na ? idx[a0 + al] : -1;
        const bool ok = ex >= 0 && ex < E;
        (void)wave_rank(ok, ex, E, lane, w, s_wc);
        __syncthreads();
        if (tid < E) {
            int s = 0;
#pragma unroll
            for (int i = 0; i < kWaves; ++i) s += s_wc[i][tid];
            s_run[tid] += s;
        }
        __syncthreads();
    }
    if (tid < E) tile_counts[static_cast<int64_t>(blockIdx.x) * E + tid] = s_run[tid];
}

// One workgroup: exclusive scan over tiles, expert by expert.
__global__ __launch_bounds__(1024) void k_scan(const int32_t* __restrict__ tc, int64_t ntiles,
                                               int E, int32_t* __restrict__ tb,
                                               int32_t* __restrict__ counts,
                                               int32_t* __restrict__ offsets) {
    __shared__ int s_wsum[16];
    __shared__ int s_tot[64];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t per = (ntiles + 1023) / 1024;
    const int64_t b0 = tid * per;
    const int64_t b1 = b0 + per < ntiles ? b0 + per : ntiles;
    for (int e = 0; e < E; ++e) {
        int s = 0;
        for (int64_t b = b0; b < b1; ++b) s += tc[b * E + e];
        int v = s;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int n = __shfl_up(v, o);
            if (lane >= o) v += n;
        }
        if (lane == 63) s_wsum[w] = v;
        __syncthreads();
        int pre = 0;
        for (int i = 0; i < w; ++i) pre += s_wsum[i];
        int run = pre + v - s;
        for (int64_t b = b0; b < b1; ++b) {
            tb[b * E + e] = run;
            run += tc[b * E + e];
        }
        if (tid == 1023) s_tot[e] = pre + v;
        __syncthreads();
    }
    if (tid == 0) {
        int o = 0;
        for (int e = 0; e < E; ++e) {
            counts[e] = s_tot[e];
            offsets[e] = o;
            o += s_tot[e];
        }
        offsets[E] = o;
    }
}

template <typename Tin>
__global__ __launch_bounds__(kRouteTile) void k_permute(
    const int32_t* __restrict__ idx, const int32_t* __restrict__ tb,
    const int32_t* __restrict__ offsets, int64_t T, int E, int k, int32_t* __restrict__ perm,
    int32_t* __restrict__ inv, const Tin* __restrict__ x, Tin* __restrict__ xperm, int D) {
    extern __shared__ int s_p[];          // [256 * k] destination of each assignment
    __shared__ int s_wc[kWaves][64];
    __shared__ int s_run[64];
    __shared__ int s_base[64];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t A = T * k;
    const int64_t a0 = static_cast<int64_t>(blockIdx.x) * kRouteTile * k;
    const int64_t na64 = A - a0 < static_cast<int64_t>(kRouteTile) * k ? A - a0
                                                                         : static_cast<int64_t>(kRouteTile) * k;
    const int na = static_cast<int>(na64);
    if (tid < E) {
        s_run[tid] = 0;
        s_base[tid] = offsets[tid] + tb[static_cast<int64_t>(blockIdx.x) * E + tid];
    }
    __syncthreads();
    for (int c = 0; c < k; ++c) {
        const int al = c * kRouteTile + tid;
        const bool valid = al < na;
        const int ex = valid ? idx[a0 + al] : -1;
        const bool ok = ex >= 0 && ex < E;    // out-of-range indices are skipped, never followed
        const int rw = wave_rank(ok, ex, E, lane, w, s_wc);
        __syncthreads();
        int p = -1;
        if (ok) {
            int r = s_run[ex] + rw;
            for (int i = 0; i < w; ++i) r += s_wc[i][ex];
            p = s_base[ex] + r;
            // a histogram that does not match idx (a broken HIST_IN_WS contract)
            // could point outside [0, T*k): such entries are dropped, never written
            if (p < 0 || static_cast<int64_t>(p) >= A) p = -1;
        }
        if (p >= 0) {
            perm[p] = static_cast<int32_t>(a0 + al);
            inv[a0 + al] = p;
            s_p[al] = p;
        } else if (valid) {
            inv[a0 + al] = -1;
            s_p[al] = -1;
        }
        __syncthreads();
        if (tid < E) {
            int s = 0;
#pragma unroll
            for (int i = 0; i < kWaves; ++i) s += s_wc[i][tid];
            s_run[tid] += s;
        }
        __syncthreads();
    }
    if (xperm != nullptr) {
        constexpr int PER16 = Elem<Tin>::per16;
        const int ppr = D / PER16;                      // 16-byte pieces per row
        const int npairs = na * ppr;
#pragma unroll 4
        for (int pr = tid; pr < npairs; pr += kRouteTile) {
            const int al = pr / ppr, pc = pr - al * ppr;
            const int p = s_p[al];
            if (p < 0) continue;
            const int64_t tok = (a0 + al) / k;
            const uint4 v = *reinterpret_cast<const uint4*>(x + tok * D + pc * PER16);
            *reinterpret_cast<uint4*>(xperm + static_cast<int64_t>(p) * D + pc * PER16) = v;
        }
    }
}

// y[t, :] = sum_j gate[t, j] * ye[inv[t*k + j], :], float32 accumulation in slot order.
template <typename T>
__global__ __launch_bounds__(256) void k_combine_gated(const T* __restrict__ ye,
                                                       const int32_t* __restrict__ inv,
                                                       const float* __restrict__ gate,
                                                       T* __restrict__ y, int64_t Tn, int D,
                                                       int k) {
    constexpr int PER16 = Elem<T>::per16;
    const int ppr = D / PER16;
    const int64_t pr = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (pr >= Tn * ppr) return;
    const int64_t t = pr / ppr;
    const int pc = static_cast<int>(pr - t * ppr);
    float acc[PER16];
#pragma unroll
    for (int u = 0; u < PER16; ++u) acc[u] = 0.0f;
    const int64_t A = Tn * k;
    for (int j = 0; j < k; ++j) {
        const int64_t p = inv[t * k + j];
        if (p < 0 || p >= A) continue;           // never follow an invalid index
        const float g = gate[t * k + j];
        const uint4 v = *reinterpret_cast<const uint4*>(ye + p * D + pc * PER16);
        T vals[PER16];
        __builtin_memcpy(vals, &v, 16);
#pragma unroll
        for (int u = 0; u < PER16; ++u) acc[u] = __builtin_fmaf(g, Elem<T>::to_f32(vals[u]), acc[u]);
    }
    T out[PER16];
#pragma unroll
    for (int u = 0; u < PER16; ++u) out[u] = Elem<T>::from_f32(acc[u]);
    uint4 o;
    __builtin_memcpy(&o, out, 16);
    *reinterpret_cast<uint4*>(y + t * D + pc * PER16) = o;
}

// y[t, :] = hsh[t, :] + sum_j hres[inv[t*k + j], :]  (float32 in, dtype out).
template <typename T>
__global__ __launch_bounds__(256) void k_combine_residual(const float* __restrict__ hsh,
                                                          const float* __restrict__ hres,
                                                          const int32_t* __restrict__ inv,
                                                          T* __restrict__ y, int64_t Tn, int D,
                                                          int k) {
    const int ppr = D / 4;                       // 4 floats per piece
    const int64_t pr = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (pr >= Tn * ppr) return;
    const int64_t t = pr / ppr;
    const int pc = static_cast<int>(pr - t * ppr);
    float4 a = *reinterpret_cast<const float4*>(hsh + t * D + pc * 4);
    const int64_t A = Tn * k;
    for (int j = 0; j < k; ++j) {
        const int64_t p = inv[t * k + j];
        if (p < 0 || p >= A) continue;
        const float4 b = *reinterpret_cast<const float4*>(hres + p * D + pc * 4);
        a.x += b.x;
        a.y += b.y;
        a.z += b.z;
        a.w += b.w;
    }
    T out[4] = {Elem<T>::from_f32(a.x), Elem<T>::from_f32(a.y), Elem<T>::from_f32(a.z),
                Elem<T>::from_f32(a.w)};
    T* dst = y + t * D + pc * 4;
#pragma unroll
    for (int u = 0; u < 4; ++u) dst[u] = out[u];
}

hipError_t launch_tile_histogram(const int32_t* idx, int64_t T, int E, int k,
                                 int32_t* tile_counts, hipStream_t st) {
    const int64_t nt = route_tiles(T);
    if (nt == 0) return hipSuccess;
    k_tile_hist<<<dim3(static_cast<unsigned>(nt)), kRouteTile, 0, st>>>(idx, T, E, k, tile_counts);
    return hipGetLastError();
}

hipError_t launch_scan(const int32_t* tile_counts, int64_t ntiles, int E, int32_t* tile_base,
                       int32_t* counts, int32_t* offsets, hipStream_t st) {
    k_scan<<<1, 1024, 0, st>>>(tile_counts, ntiles, E, tile_base, counts, offsets);
    return hipGetLastError();
}

hipError_t launch_permute(int dtype, const int32_t* idx, const int32_t* tile_base,
                          const int32_t* offsets, int64_t T, int E, int k, int32_t* perm,
                          int32_t* inv, const void* x, void* xperm, int D, hipStream_t st) {
    const int64_t nt = route_tiles(T);
    if (nt == 0) return hipSuccess;
    const size_t shm = sizeof(int) * static_cast<size_t>(kRouteTile) * k;
    if (dtype == 0)
        k_permute<float><<<dim3(static_cast<unsigned>(nt)), kRouteTile, shm, st>>>(
            idx, tile_base, offsets, T, E, k, perm, inv, static_cast<const float*>(x),
            static_cast<float*>(xperm), D);
    else
        k_permute<bf16_bits><<<dim3(static_cast<unsigned>(nt)), kRouteTile, shm, st>>>(
            idx, tile_base, offsets, T, E, k, perm, inv, static_cast<const bf16_bits*>(x),
            static_cast<bf16_bits*>(xperm), D);
    return hipGetLastError();
}

hipError_t launch_combine_gated(int dtype, const void* ye, const int32_t* inv, const float* gate,
                                void* y, int64_t T, int D, int k, hipStream_t st) {
    const int per16 = dtype == 0 ? 4 : 8;
    const int64_t n = T * (D / per16);
    if (n == 0) return hipSuccess;
    const unsigned blocks = static_cast<unsigned>((n + 255) / 256);
    if (dtype == 0)
        k_combine_gated<float><<<blocks, 256, 0, st>>>(static_cast<const float*>(ye), inv, gate,
                                                        static_cast<float*>(y), T, D, k);
    else
        k_combine_gated<bf16_bits><<<blocks, 256, 0, st>>>(
            static_cast<const bf16_bits*>(ye), inv, gate, static_cast<bf16_bits*>(y), T, D, k);
    return hipGetLastError();
}

hipError_t launch_combine_residual(int dtype, const float* hsh, const float* hres,
                                   const int32_t* inv, void* y, int64_t T, int D, int k,
                                   hipStream_t st) {
    const int64_t n = T * (D / 4);
    if (n == 0) return hipSuccess;
    const unsigned blocks = static_cast<unsigned>((n + 255) / 256);
    if (dtype == 0)
        k_combine_residual<float><<<blocks, 256, 0, st>>>(hsh, hres, inv, static_cast<float*>(y),
                                                           T, D, k);
    else
        k_combine_residual<bf16_bits><<<blocks, 256, 0, st>>>(hsh, hres, inv,
                                                               static_cast<bf16_bits*>(y), T, D, k);
    return hipGetLastError();
}

}  // namespace clearmoe
