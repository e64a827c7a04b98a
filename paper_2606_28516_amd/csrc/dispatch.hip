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

// Expert histogram of one tile of TILE tokens (= TILE * k assignments), one
// workgroup of TILE threads per tile.
template <int TILE>
__global__ __launch_bounds__(TILE) void k_tile_hist(const int32_t* __restrict__ idx, int64_t T,
                                                     int E, int k,
                                                     int32_t* __restrict__ tile_counts) {
    constexpr int kW = TILE / 64;
    __shared__ int s_wc[kW][64];
    __shared__ int s_run[64];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t A = T * k;
    const int64_t a0 = static_cast<int64_t>(blockIdx.x) * TILE * k;
    const int64_t na64 = A - a0 < static_cast<int64_t>(TILE) * k ? A - a0 : static_cast<int64_t>(TILE) * k;
    const int na = static_cast<int>(na64);
    if (tid < E) s_run[tid] = 0;
    __syncthreads();
    for (int c = 0; c < k; ++c) {
        const int al = c * TILE + tid;
        const int ex = al < na ? idx[a0 + al] : -1;
        const bool ok = ex >= 0 && ex < E;
        (void)wave_rank(ok, ex, E, lane, w, s_wc);
        __syncthreads();
        if (tid < E) {
            int s = 0;
#pragma unroll
            for (int i = 0; i < kW; ++i) s += s_wc[i][tid];
            s_run[tid] += s;
        }
        __syncthreads();
    }
    if (tid < E) tile_counts[static_cast<int64_t>(blockIdx.x) * E + tid] = s_run[tid];
}

// Exclusive scan over tiles of every expert column, in chunks of kScanChunk
// tiles: workgroup c scans tiles [c kScanChunk, (c + 1) kScanChunk), one per
// thread, EP expert columns at a time (a thread holds EP counts in registers;
// the wave scans them with shuffles, wave totals meet in LDS), and writes the
// within-chunk exclusive prefixes tb and the chunk's totals.  The
// permutation adds the chunk prefixes, so every chunk runs in parallel.
constexpr int kScanChunk = 256;

template <int EP>
__global__ __launch_bounds__(kScanChunk) void k_scan(const int32_t* __restrict__ tc, int64_t ntiles,
                                                     int E, int32_t* __restrict__ tb,
                                                     int32_t* __restrict__ chunk_tot) {
    constexpr int kW = kScanChunk / 64;
    __shared__ int s_wsum[kW][EP];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t b = static_cast<int64_t>(blockIdx.x) * kScanChunk + tid;
    const bool in = b < ntiles;
    for (int e0 = 0; e0 < E; e0 += EP) {
        int v[EP], c[EP];
#pragma unroll
        for (int e = 0; e < EP; ++e) {
            c[e] = (in && e0 + e < E) ? tc[b * E + e0 + e] : 0;
            v[e] = c[e];
        }
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
#pragma unroll
            for (int e = 0; e < EP; ++e) {
                const int n = __shfl_up(v[e], o);
                if (lane >= o) v[e] += n;
            }
        }
        if (e0 > 0) __syncthreads();             // the previous block's sums are read
        if (lane == 63) {
#pragma unroll
            for (int e = 0; e < EP; ++e) s_wsum[w][e] = v[e];
        }
        __syncthreads();
#pragma unroll
        for (int e = 0; e < EP; ++e) {
            int pre = 0;
            for (int i = 0; i < w; ++i) pre += s_wsum[i][e];
            if (in && e0 + e < E) tb[b * E + e0 + e] = pre + v[e] - c[e];
        }
        if (tid < EP && e0 + tid < E) {
            int sum = 0;
#pragma unroll
            for (int i = 0; i < kW; ++i) sum += s_wsum[i][tid];
            chunk_tot[static_cast<int64_t>(blockIdx.x) * E + e0 + tid] = sum;
        }
    }
}

// Stable permutation, one workgroup per 256 tokens.  Tile bases come either
// from the scan kernel (tile_base + offsets, 256-token tiles) or, when
// tile_counts is given (small histograms), from an inline scan: every
// workgroup sums the histogram columns itself (LDS integer atomics: exact and
// order independent; the histogram tiles hold htile tokens, 64 or 256, so a
// workgroup's tokens start at histogram tile blockIdx * 256 / htile) and
// workgroup 0 publishes counts and offsets.
template <typename Tin>
__global__ __launch_bounds__(kRouteTile) void k_permute(
    const int32_t* __restrict__ idx, const int32_t* __restrict__ tb,
    int32_t* __restrict__ offsets, const int32_t* __restrict__ tile_counts,
    int32_t* __restrict__ counts, int64_t T, int E, int k, int32_t* __restrict__ perm,
    int32_t* __restrict__ inv, const Tin* __restrict__ x, Tin* __restrict__ xperm, int D,
    int htile, const int32_t* __restrict__ chunk_tot) {
    extern __shared__ int s_p[];          // [256 * k] destination of each assignment
    __shared__ int s_wc[kWaves][64];
    __shared__ int s_run[64];
    __shared__ int s_base[64];
    __shared__ int s_pre[64], s_tot[64];
    __shared__ int s_total;               // assignments that have an expert
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t A = T * k;
    const int64_t a0 = static_cast<int64_t>(blockIdx.x) * kRouteTile * k;
    const int64_t na64 = A - a0 < static_cast<int64_t>(kRouteTile) * k ? A - a0
                                                                         : static_cast<int64_t>(kRouteTile) * k;
    const int na = static_cast<int>(na64);
    if (tile_counts != nullptr) {
        if (tid < E) {
            s_pre[tid] = 0;
            s_tot[tid] = 0;
        }
        __syncthreads();
        const int64_t nt = (T + htile - 1) / htile;
        const int64_t first = static_cast<int64_t>(blockIdx.x) * (kRouteTile / htile);
        // thread tid sums, for expert tid % E, the tiles tid / E + G i in
        // registers (coalesced reads), then adds its two sums into LDS: one
        // atomic per thread instead of one per histogram entry
        const int G = kRouteTile / E;                  // threads per expert
        if (tid < G * E) {
            const int e = tid % E;
            int tot = 0, pre = 0;
            for (int64_t b = tid / E; b < nt; b += G) {
                const int c = tile_counts[b * E + e];
                tot += c;
                pre += b < first ? c : 0;
            }
            atomicAdd(&s_tot[e], tot);
            atomicAdd(&s_pre[e], pre);
        }
        __syncthreads();
        if (tid == 0) {
            int o = 0;
            for (int e = 0; e < E; ++e) {
                s_base[e] = o + s_pre[e];
                if (blockIdx.x == 0) {
                    counts[e] = s_tot[e];
                    offsets[e] = o;
                }
                o += s_tot[e];
            }
            if (blockIdx.x == 0) offsets[E] = o;
            s_total = o;
        }
        if (tid < E) s_run[tid] = 0;
    } else {
        // tile bases from the chunked scan: earlier chunks' totals plus the
        // prefix within this tile's chunk; offsets from the grand totals
        if (tid < E) {
            s_pre[tid] = 0;
            s_tot[tid] = 0;
        }
        __syncthreads();
        const int64_t nchunks = (route_tiles(T) + kScanChunk - 1) / kScanChunk;
        const int64_t mychunk = static_cast<int64_t>(blockIdx.x) / kScanChunk;
        const int G = kRouteTile / E;
        if (tid < G * E) {
            const int e = tid % E;
            int tot = 0, pre = 0;
            for (int64_t c = tid / E; c < nchunks; c += G) {
                const int v = chunk_tot[c * E + e];
                tot += v;
                pre += c < mychunk ? v : 0;
            }
            atomicAdd(&s_tot[e], tot);
            atomicAdd(&s_pre[e], pre);
        }
        __syncthreads();
        if (tid == 0) {
            int o = 0;
            for (int e = 0; e < E; ++e) {
                s_base[e] = o + s_pre[e] + tb[static_cast<int64_t>(blockIdx.x) * E + e];
                if (blockIdx.x == 0) {
                    counts[e] = s_tot[e];
                    offsets[e] = o;
                }
                o += s_tot[e];
            }
            if (blockIdx.x == 0) offsets[E] = o;
            s_total = o;
        }
        if (tid < E) s_run[tid] = 0;
    }
    __syncthreads();
    // Empty slots (index -1) are in no sub-batch: perm ends with -1 entries
    // after the offsets[E] real assignments.
    for (int64_t i = static_cast<int64_t>(s_total) + static_cast<int64_t>(blockIdx.x) * kRouteTile + tid;
         i < A; i += static_cast<int64_t>(gridDim.x) * kRouteTile)
        if (i >= 0) perm[i] = -1;
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
        // Row copy: 16-byte pieces, eight per thread per round (all loads
        // issued before the stores; measured against 4 and 16 at 2^20 tokens);
        // the destination rows are written once and read later by another
        // kernel, so the stores bypass the caches.
        constexpr int PER16 = Elem<Tin>::per16;
        constexpr int U = 8;
        const int ppr = D / PER16;                      // 16-byte pieces per row
        const int npairs = na * ppr;
        for (int base = 0; base < npairs; base += U * kRouteTile) {
            u32x4 v[U];
            int dp[U], dc[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int pr = base + u * kRouteTile + tid;
                dp[u] = -1;
                dc[u] = 0;
                if (pr < npairs) {
                    const int al = pr / ppr, pc = pr - al * ppr;
                    const int p = s_p[al];
                    if (p >= 0) {
                        const int64_t tok = (a0 + al) / k;
                        v[u] = *reinterpret_cast<const u32x4*>(x + tok * D + pc * PER16);
                        dp[u] = p;
                        dc[u] = pc;
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
                if (dp[u] >= 0)
                    __builtin_nontemporal_store(
                        v[u], reinterpret_cast<u32x4*>(xperm + static_cast<int64_t>(dp[u]) * D +
                                                       dc[u] * PER16));
        }
    }
}

constexpr int kCombineU = 4;   // 16-byte output pieces per thread

// y[t, :] = sum_j gate[t, j] * ye[inv[t*k + j], :], float32 accumulation in
// slot order.  A workgroup covers 256*U consecutive 16-byte pieces of y, a
// thread U of them (stride 256, so each load instruction is coalesced).
template <typename T>
__global__ __launch_bounds__(256) void k_combine_gated(const T* __restrict__ ye,
                                                       const int32_t* __restrict__ inv,
                                                       const float* __restrict__ gate,
                                                       T* __restrict__ y, int64_t Tn, int D,
                                                       int k) {
    constexpr int PER16 = Elem<T>::per16;
    const int ppr = D / PER16;
    const int64_t n = Tn * ppr, A = Tn * k;
    const int64_t base = static_cast<int64_t>(blockIdx.x) * 256 * kCombineU + threadIdx.x;
    float acc[kCombineU][PER16];
#pragma unroll
    for (int u = 0; u < kCombineU; ++u)
#pragma unroll
        for (int i = 0; i < PER16; ++i) acc[u][i] = 0.0f;
    for (int j = 0; j < k; ++j) {
        u32x4 v[kCombineU];
        float g[kCombineU];
#pragma unroll
        for (int u = 0; u < kCombineU; ++u) {
            const int64_t pr = base + u * 256;
            g[u] = 0.0f;
            v[u] = u32x4{0u, 0u, 0u, 0u};
            if (pr < n) {
                const int64_t t = pr / ppr, pc = pr - t * ppr;
                const int64_t p = inv[t * k + j];
                if (p >= 0 && p < A) {               // never follow an invalid index
                    g[u] = gate[t * k + j];
                    v[u] = *reinterpret_cast<const u32x4*>(ye + p * D + pc * PER16);
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kCombineU; ++u) {
            T vals[PER16];
            __builtin_memcpy(vals, &v[u], 16);
#pragma unroll
            for (int i = 0; i < PER16; ++i)
                acc[u][i] = __builtin_fmaf(g[u], Elem<T>::to_f32(vals[i]), acc[u][i]);
        }
    }
#pragma unroll
    for (int u = 0; u < kCombineU; ++u) {
        const int64_t pr = base + u * 256;
        if (pr >= n) continue;
        T out[PER16];
#pragma unroll
        for (int i = 0; i < PER16; ++i) out[i] = Elem<T>::from_f32(acc[u][i]);
        u32x4 o;
        __builtin_memcpy(&o, out, 16);
        const int64_t t = pr / ppr, pc = pr - t * ppr;
        *reinterpret_cast<u32x4*>(y + t * D + pc * PER16) = o;
    }
}

// y[t, :] = hsh[t, :] + sum_j hres[inv[t*k + j], :]  (float32 in, dtype out);
// 4-float pieces, U per thread as above.
template <typename T>
__global__ __launch_bounds__(256) void k_combine_residual(const float* __restrict__ hsh,
                                                          const float* __restrict__ hres,
                                                          const int32_t* __restrict__ inv,
                                                          T* __restrict__ y, int64_t Tn, int D,
                                                          int k, int64_t hres_rows) {
    const int ppr = D / 4;
    const int64_t n = Tn * ppr, A = hres_rows;
    const int64_t base = static_cast<int64_t>(blockIdx.x) * 256 * kCombineU + threadIdx.x;
    float4 a[kCombineU];
#pragma unroll
    for (int u = 0; u < kCombineU; ++u) {
        const int64_t pr = base + u * 256;
        a[u] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (pr < n) {
            const int64_t t = pr / ppr, pc = pr - t * ppr;
            a[u] = *reinterpret_cast<const float4*>(hsh + t * D + pc * 4);
        }
    }
    for (int j = 0; j < k; ++j) {
        float4 bv[kCombineU];
#pragma unroll
        for (int u = 0; u < kCombineU; ++u) {
            const int64_t pr = base + u * 256;
            bv[u] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (pr < n) {
                const int64_t t = pr / ppr, pc = pr - t * ppr;
                const int64_t p = inv[t * k + j];
                if (p >= 0 && p < A) bv[u] = *reinterpret_cast<const float4*>(hres + p * D + pc * 4);
            }
        }
#pragma unroll
        for (int u = 0; u < kCombineU; ++u) {
            a[u].x += bv[u].x;
            a[u].y += bv[u].y;
            a[u].z += bv[u].z;
            a[u].w += bv[u].w;
        }
    }
#pragma unroll
    for (int u = 0; u < kCombineU; ++u) {
        const int64_t pr = base + u * 256;
        if (pr >= n) continue;
        const int64_t t = pr / ppr, pc = pr - t * ppr;
        T* dst = y + t * D + pc * 4;
        dst[0] = Elem<T>::from_f32(a[u].x);
        dst[1] = Elem<T>::from_f32(a[u].y);
        dst[2] = Elem<T>::from_f32(a[u].z);
        dst[3] = Elem<T>::from_f32(a[u].w);
    }
}

hipError_t launch_tile_histogram(const int32_t* idx, int64_t T, int E, int k,
                                 int32_t* tile_counts, hipStream_t st) {
    const int64_t nt = hist_tiles(T, E);
    if (nt == 0) return hipSuccess;
    if (hist_tile(T, E) == kSmallTile)
        launch_kernel(k_tile_hist<kSmallTile>, dim3(static_cast<unsigned>(nt)), kSmallTile, 0, st, idx, T, E, k,
                                                                                        tile_counts);
    else
        launch_kernel(k_tile_hist<kRouteTile>, dim3(static_cast<unsigned>(nt)), kRouteTile, 0, st, idx, T, E, k,
                                                                                        tile_counts);
    return hipGetLastError();
}

int64_t scan_chunks(int64_t ntiles) { return (ntiles + kScanChunk - 1) / kScanChunk; }

hipError_t launch_scan(const int32_t* tile_counts, int64_t ntiles, int E, int32_t* tile_base,
                       int32_t* chunk_tot, hipStream_t st) {
    const dim3 grid(static_cast<unsigned>(scan_chunks(ntiles)));
    if (ntiles == 0) return hipSuccess;
    // 16 columns at a time beyond 8 experts (64 per pass spilled registers)
    if (E <= 8)
        launch_kernel(k_scan<8>, grid, kScanChunk, 0, st, tile_counts, ntiles, E, tile_base, chunk_tot);
    else
        launch_kernel(k_scan<16>, grid, kScanChunk, 0, st, tile_counts, ntiles, E, tile_base, chunk_tot);
    return hipGetLastError();
}

hipError_t launch_permute(int dtype, const int32_t* idx, const int32_t* tile_base,
                          const int32_t* chunk_tot, int32_t* offsets, const int32_t* tile_counts,
                          int32_t* counts, int64_t T, int E, int k, int32_t* perm, int32_t* inv,
                          const void* x, void* xperm, int D, hipStream_t st) {
    const int64_t nt = route_tiles(T);
    if (nt == 0) return hipSuccess;
    const size_t shm = sizeof(int) * static_cast<size_t>(kRouteTile) * k;
    const int htile = hist_tile(T, E);
    if (dtype == 0)
        launch_kernel(k_permute<float>, dim3(static_cast<unsigned>(nt)), kRouteTile, shm, st,
            idx, tile_base, offsets, tile_counts, counts, T, E, k, perm, inv,
            static_cast<const float*>(x), static_cast<float*>(xperm), D, htile, chunk_tot);
    else
        launch_kernel(k_permute<bf16_bits>, dim3(static_cast<unsigned>(nt)), kRouteTile, shm, st,
            idx, tile_base, offsets, tile_counts, counts, T, E, k, perm, inv,
            static_cast<const bf16_bits*>(x), static_cast<bf16_bits*>(xperm), D, htile, chunk_tot);
    return hipGetLastError();
}

hipError_t launch_combine_gated(int dtype, const void* ye, const int32_t* inv, const float* gate,
                                void* y, int64_t T, int D, int k, hipStream_t st) {
    const int per16 = dtype == 0 ? 4 : 8;
    const int64_t n = T * (D / per16);
    if (n == 0) return hipSuccess;
    const unsigned blocks = static_cast<unsigned>((n + 256 * kCombineU - 1) / (256 * kCombineU));
    if (dtype == 0)
        launch_kernel(k_combine_gated<float>, blocks, 256, 0, st, static_cast<const float*>(ye), inv, gate,
                                                        static_cast<float*>(y), T, D, k);
    else
        launch_kernel(k_combine_gated<bf16_bits>, blocks, 256, 0, st,
            static_cast<const bf16_bits*>(ye), inv, gate, static_cast<bf16_bits*>(y), T, D, k);
    return hipGetLastError();
}

// Row width D that is not a multiple of the elements of a 16-byte piece:
// the same row gather and gated combine one element per thread (the
// combine's arithmetic is the 16-byte kernel's: float32 fma in slot order
// from 0, one rounding to the storage type).
template <typename T>
__global__ __launch_bounds__(256) void k_gather_rows_elem(const T* __restrict__ x,
                                                          const int32_t* __restrict__ perm,
                                                          const int32_t* __restrict__ nreal,
                                                          int64_t A, int k, int D,
                                                          T* __restrict__ xperm) {
    int64_t rows = *nreal;                        // rows past offsets[E] are not written
    rows = rows < 0 ? 0 : (rows > A ? A : rows);
    const int64_t n = rows * D;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t p = i / D, c = i - p * D;
        const int64_t a = perm[p];
        if (a >= 0 && a < A) xperm[i] = x[(a / k) * D + c];
    }
}

template <typename T>
__global__ __launch_bounds__(256) void k_combine_gated_elem(const T* __restrict__ ye,
                                                            const int32_t* __restrict__ inv,
                                                            const float* __restrict__ gate,
                                                            T* __restrict__ y, int64_t Tn, int D,
                                                            int k) {
    const int64_t n = Tn * D, A = Tn * k;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t t = i / D, c = i - t * D;
        float acc = 0.0f;
        for (int j = 0; j < k; ++j) {
            const int64_t p = inv[t * k + j];
            if (p >= 0 && p < A)                  // never follow an invalid index
                acc = __builtin_fmaf(gate[t * k + j], Elem<T>::to_f32(ye[p * D + c]), acc);
        }
        y[i] = Elem<T>::from_f32(acc);
    }
}

static unsigned elem_blocks(int64_t n) {
    const int64_t b = (n + 255) / 256;
    return static_cast<unsigned>(b < 8192 ? b : 8192);
}

hipError_t launch_gather_rows_elem(int dtype, const void* x, const int32_t* perm,
                                   const int32_t* nreal, int64_t A, int k, int D, void* xperm,
                                   hipStream_t st) {
    if (A * D == 0) return hipSuccess;
    if (dtype == 0)
        launch_kernel(k_gather_rows_elem<float>, elem_blocks(A * D), 256, 0, st,
                      static_cast<const float*>(x), perm, nreal, A, k, D, static_cast<float*>(xperm));
    else
        launch_kernel(k_gather_rows_elem<bf16_bits>, elem_blocks(A * D), 256, 0, st,
                      static_cast<const bf16_bits*>(x), perm, nreal, A, k, D,
                      static_cast<bf16_bits*>(xperm));
    return hipGetLastError();
}

hipError_t launch_combine_gated_elem(int dtype, const void* ye, const int32_t* inv,
                                     const float* gate, void* y, int64_t T, int D, int k,
                                     hipStream_t st) {
    if (T * D == 0) return hipSuccess;
    if (dtype == 0)
        launch_kernel(k_combine_gated_elem<float>, elem_blocks(T * D), 256, 0, st,
                      static_cast<const float*>(ye), inv, gate, static_cast<float*>(y), T, D, k);
    else
        launch_kernel(k_combine_gated_elem<bf16_bits>, elem_blocks(T * D), 256, 0, st,
                      static_cast<const bf16_bits*>(ye), inv, gate, static_cast<bf16_bits*>(y), T,
                      D, k);
    return hipGetLastError();
}

hipError_t launch_combine_residual(int dtype, const float* hsh, const float* hres,
                                   const int32_t* inv, void* y, int64_t T, int D, int k,
                                   int64_t hres_rows, hipStream_t st) {
    const int64_t n = T * (D / 4);
    if (n == 0) return hipSuccess;
    const unsigned blocks = static_cast<unsigned>((n + 256 * kCombineU - 1) / (256 * kCombineU));
    if (dtype == 0)
        launch_kernel(k_combine_residual<float>, blocks, 256, 0, st, hsh, hres, inv, static_cast<float*>(y),
                                                           T, D, k, hres_rows);
    else
        launch_kernel(k_combine_residual<bf16_bits>, blocks, 256, 0, st,
            hsh, hres, inv, static_cast<bf16_bits*>(y), T, D, k, hres_rows);
    return hipGetLastError();
}

// out = x + f element by element (float32 sum, one rounding to the storage
// type): the skip connection around a stack's FFN layer.  16-byte pieces.
template <typename T>
__global__ __launch_bounds__(256) void k_residual_add(const T* __restrict__ x,
                                                      const T* __restrict__ f,
                                                      T* __restrict__ out, int64_t n16) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i >= n16) return;
    constexpr int P = Elem<T>::per16;
    const uint4 xa = reinterpret_cast<const uint4*>(x)[i];
    const uint4 fa = reinterpret_cast<const uint4*>(f)[i];
    const T* xv = reinterpret_cast<const T*>(&xa);
    const T* fv = reinterpret_cast<const T*>(&fa);
    float v[P];
#pragma unroll
    for (int j = 0; j < P; ++j) v[j] = Elem<T>::to_f32(xv[j]) + Elem<T>::to_f32(fv[j]);
    uint4 o;
    T* ov = reinterpret_cast<T*>(&o);
#pragma unroll
    for (int j = 0; j < P; ++j) ov[j] = Elem<T>::from_f32(v[j]);
    reinterpret_cast<uint4*>(out)[i] = o;
}

hipError_t launch_residual_add(int dtype, const void* x, const void* f, void* out, int64_t T, int D,
                               hipStream_t st) {
    const int per16 = dtype == 0 ? 4 : 8;
    const int64_t n16 = T * (D / per16);
    if (n16 == 0) return hipSuccess;
    const unsigned blocks = static_cast<unsigned>((n16 + 255) / 256);
    if (dtype == 0)
        launch_kernel(k_residual_add<float>, blocks, 256, 0, st, static_cast<const float*>(x),
                      static_cast<const float*>(f), static_cast<float*>(out), n16);
    else
        launch_kernel(k_residual_add<bf16_bits>, blocks, 256, 0, st, static_cast<const bf16_bits*>(x),
                      static_cast<const bf16_bits*>(f), static_cast<bf16_bits*>(out), n16);
    return hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void k_pad_copy(const T* __restrict__ src, T* __restrict__ dst,
                                                  int64_t batches, int64_t srows, int64_t scols,
                                                  int64_t drows, int64_t dcols) {
    const int64_t n = batches * drows * dcols;
    for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n;
         i += static_cast<int64_t>(gridDim.x) * blockDim.x) {
        const int64_t c = i % dcols, br = i / dcols;
        const int64_t r = br % drows, b = br / drows;
        dst[i] = (r < srows && c < scols) ? src[(b * srows + r) * scols + c] : T(0);
    }
}

hipError_t launch_pad_copy(int elem_bytes, const void* src, void* dst, int64_t batches, int64_t srows,
                           int64_t scols, int64_t drows, int64_t dcols, hipStream_t st) {
    if (batches < 0 || srows < 0 || scols < 0 || drows < 0 || dcols < 0) return hipErrorInvalidValue;
    const int64_t n = batches * drows * dcols;
    if (n == 0) return hipSuccess;
    if (src == nullptr || dst == nullptr) return hipErrorInvalidValue;
    const int64_t b = (n + 255) / 256;
    const unsigned blocks = static_cast<unsigned>(b < 8192 ? b : 8192);
    if (elem_bytes == 4)
        launch_kernel(k_pad_copy<uint32_t>, blocks, 256, 0, st, static_cast<const uint32_t*>(src),
                      static_cast<uint32_t*>(dst), batches, srows, scols, drows, dcols);
    else if (elem_bytes == 2)
        launch_kernel(k_pad_copy<uint16_t>, blocks, 256, 0, st, static_cast<const uint16_t*>(src),
                      static_cast<uint16_t*>(dst), batches, srows, scols, drows, dcols);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

// Pair keys of a top-2 routing (see launch_pair_key): a token with one expert
// e gets key e and gates (gate of e, 0); one with experts a < b gets key
// E + (number of the pair (a, b) in lexicographic order) and gates (gate of
// a, gate of b); one with none gets -1 (no segment).  Workgroup i takes the
// TILE tokens of histogram tile i and also writes the tile's key counts, so
// the dispatch over keys needs no histogram pass of its own.
template <int TILE>
__global__ __launch_bounds__(TILE) void k_pair_key(const int32_t* __restrict__ idx,
                                                   const float* __restrict__ gate, int64_t T, int E,
                                                   int nkeys, int32_t* __restrict__ key,
                                                   float* __restrict__ ga, float* __restrict__ gb,
                                                   int32_t* __restrict__ tile_counts) {
    constexpr int kW = TILE / 64;
    __shared__ int s_wc[kW][64];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t t = static_cast<int64_t>(blockIdx.x) * TILE + tid;
    int32_t kk = -1;
    if (t < T) {
        // idx and gate may be only 4-byte aligned (caller arrays): two loads each
        const int2 e = make_int2(idx[2 * t], idx[2 * t + 1]);
        const float2 g = make_float2(gate[2 * t], gate[2 * t + 1]);
        const bool v0 = e.x >= 0 && e.x < E, v1 = e.y >= 0 && e.y < E;
        float2 o = make_float2(0.0f, 0.0f);
        if (v0 && v1 && e.x != e.y) {
            const bool lo0 = e.x < e.y;
            const int a = lo0 ? e.x : e.y, b = lo0 ? e.y : e.x;
            kk = E + a * (2 * E - a - 1) / 2 + (b - a - 1);
            o = lo0 ? g : make_float2(g.y, g.x);
        } else if (v0 || v1) {
            kk = v0 ? e.x : e.y;
            o = make_float2(v0 ? g.x : g.y, 0.0f);
        }
        key[t] = kk;
        ga[t] = o.x;
        gb[t] = o.y;
    }
    (void)wave_rank(kk >= 0, kk, nkeys, lane, w, s_wc);
    __syncthreads();
    if (tid < nkeys) {
        int c = 0;
#pragma unroll
        for (int i = 0; i < kW; ++i) c += s_wc[i][tid];
        tile_counts[static_cast<int64_t>(blockIdx.x) * nkeys + tid] = c;
    }
}

hipError_t launch_pair_key(const int32_t* idx, const float* gate, int64_t T, int E, int32_t* key,
                           float* ga, float* gb, int32_t* tile_counts, hipStream_t st) {
    const int nkeys = pair_keys(E);
    if (nkeys > kPairMaxKeys) return hipErrorInvalidValue;
    const int64_t nt = hist_tiles(T, nkeys);
    if (nt == 0) return hipSuccess;
    if (hist_tile(T, nkeys) == kSmallTile)
        launch_kernel(k_pair_key<kSmallTile>, dim3(static_cast<unsigned>(nt)), kSmallTile, 0, st, idx, gate, T,
                      E, nkeys, key, ga, gb, tile_counts);
    else
        launch_kernel(k_pair_key<kRouteTile>, dim3(static_cast<unsigned>(nt)), kRouteTile, 0, st, idx, gate, T,
                      E, nkeys, key, ga, gb, tile_counts);
    return hipGetLastError();
}

// Padded batches: expert e owns rows [e C, e C + C) of the padded order.
//   perm_pad[e C + i] = perm[offsets[e] + i] for i < counts[e], else -1;
//   inv_pad[a] = e C + (inv[a] - offsets[e]) with e = idx[a];
//   seg[e] = e C (e = 0..E).
__global__ __launch_bounds__(256) void k_pad_index(const int32_t* __restrict__ idx,
                                                   const int32_t* __restrict__ counts,
                                                   const int32_t* __restrict__ offsets,
                                                   const int32_t* __restrict__ perm,
                                                   const int32_t* __restrict__ inv, int64_t A, int E,
                                                   int64_t C, int32_t* __restrict__ perm_pad,
                                                   int32_t* __restrict__ inv_pad,
                                                   int32_t* __restrict__ seg) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    const int64_t npad = static_cast<int64_t>(E) * C;
    if (i < npad) {
        const int e = static_cast<int>(i / C);
        const int64_t r = i - static_cast<int64_t>(e) * C;
        perm_pad[i] = r < counts[e] ? perm[offsets[e] + r] : -1;
    }
    if (i < A) {
        const int e = idx[i];
        inv_pad[i] = (e >= 0 && e < E) ? static_cast<int32_t>(static_cast<int64_t>(e) * C + inv[i] - offsets[e])
                                       : -1;
    }
    if (i <= E) seg[i] = static_cast<int32_t>(i * C);
}

hipError_t launch_pad_index(const int32_t* idx, const int32_t* counts, const int32_t* offsets,
                            const int32_t* perm, const int32_t* inv, int64_t A, int E, int64_t C,
                            int32_t* perm_pad, int32_t* inv_pad, int32_t* seg, hipStream_t st) {
    int64_t n = static_cast<int64_t>(E) * C;
    if (A > n) n = A;
    if (E + 1 > n) n = E + 1;
    const unsigned blocks = static_cast<unsigned>((n + 255) / 256);
    launch_kernel(k_pad_index, blocks, 256, 0, st, idx, counts, offsets, perm, inv, A, E, C, perm_pad, inv_pad, seg);
    return hipGetLastError();
}

}  // namespace clearmoe
