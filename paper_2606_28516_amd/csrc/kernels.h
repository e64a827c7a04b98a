// Internal declarations of the CLEAR-MoE HIP kernels (gfx950) and their host
// launchers.  Nothing here is part of the public C ABI (include/clearmoe.h).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace clearmoe {

// ---------------------------------------------------------------------------
// Element types.  bfloat16 is carried as raw 16-bit patterns in memory.
// ---------------------------------------------------------------------------
typedef uint16_t bf16_bits;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_to_f32(bf16_bits b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// float -> bfloat16, round to nearest even (NaN kept quiet).
__device__ __forceinline__ bf16_bits f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<bf16_bits>((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<bf16_bits>(u >> 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
    static constexpr int per16 = 4;                 // elements per 16-byte piece
    __device__ static float load(const float* p, int64_t i) { return p[i]; }
    __device__ static float to_f32(float v) { return v; }
    __device__ static float from_f32(float v) { return v; }
};
template <> struct Elem<bf16_bits> {
    static constexpr int per16 = 8;
    __device__ static float load(const bf16_bits* p, int64_t i) { return bf16_to_f32(p[i]); }
    __device__ static float to_f32(bf16_bits v) { return bf16_to_f32(v); }
    __device__ static bf16_bits from_f32(float v) { return f32_to_bf16(v); }
};

// Exact-erf GELU in float32 (device erff).
__device__ __forceinline__ float gelu_erf(float v) {
    return 0.5f * v * (1.0f + erff(v * 0.70710678118654752440f));
}

// ---------------------------------------------------------------------------
// Tiling constants shared by host and device code.
// ---------------------------------------------------------------------------
constexpr int kRouteTile = 256;      // tokens per routing / dispatch tile (one per thread)

__host__ __device__ inline int64_t route_tiles(int64_t T) { return (T + kRouteTile - 1) / kRouteTile; }

// ---------------------------------------------------------------------------
// Host launchers (return hipError_t of the launch).
// ---------------------------------------------------------------------------
// Router logits (float32 MFMA, certified; double recompute of near ties),
// top-k, gates, per-tile expert histogram (tile_counts may be NULL).
hipError_t launch_route(int dtype, const void* x, const void* Wg, const float* bg, int64_t T,
                        int D, int E, int k, int32_t* idx, float* gate, int32_t* tile_counts,
                        hipStream_t st);
// Per-tile expert histogram of an index array.
hipError_t launch_tile_histogram(const int32_t* idx, int64_t T, int E, int k,
                                 int32_t* tile_counts, hipStream_t st);
// Exclusive scan of tile histograms: tile_base[b][e] = sum_{b'<b} tile_counts[b'][e];
// counts[e] = column sums; offsets[e] = exclusive scan of counts (offsets[E] = total).
hipError_t launch_scan(const int32_t* tile_counts, int64_t ntiles, int E, int32_t* tile_base,
                       int32_t* counts, int32_t* offsets, hipStream_t st);
// Stable permutation (and optional row copy x -> xperm).  With tile_counts
// non-NULL the tile scan is done inline (tile_base unused) and counts/offsets
// are written; otherwise tile_base/offsets come from launch_scan.
hipError_t launch_permute(int dtype, const int32_t* idx, const int32_t* tile_base,
                          int32_t* offsets, const int32_t* tile_counts, int32_t* counts,
                          int64_t T, int E, int k, int32_t* perm, int32_t* inv, const void* x,
                          void* xperm, int D, hipStream_t st);
// Largest tile histogram (tiles x experts) scanned inline by the permutation.
constexpr int64_t kInlineScanMax = 8192;
// y[t] = sum_j gate[t,j] ye[inv[t*k+j]]  (ye, y in dtype).
hipError_t launch_combine_gated(int dtype, const void* ye, const int32_t* inv, const float* gate,
                                void* y, int64_t T, int D, int k, hipStream_t st);
// y[t] = hsh[t] + sum_j hres[inv[t*k+j]]  (hsh, hres float32; y in dtype).
hipError_t launch_combine_residual(int dtype, const float* hsh, const float* hres,
                                   const int32_t* inv, void* y, int64_t T, int D, int k,
                                   hipStream_t st);

// NT GEMM  C[crow(m), n] = epi( sum_k A[arow(m), k] B_seg(m)[n, k] ).
// B may come in two parts: rows n >= n_split from B1 (row n - n_split), or
// columns k >= k_split from B1 (column k - k_split); each part has its own
// per-segment stride (0 = shared by all segments).
struct GemmDesc {
    const void* A;            // [*, K] in dtype, row stride lda (elements)
    int64_t lda;
    const int32_t* a_rows;    // optional gather: A row = a_rows[m] / a_div
    int a_div;
    const void* B;            // part 0: [N, K] per segment, row stride ldb
    int64_t ldb;
    int64_t b_seg_stride;     // elements between segments (0 = shared)
    const void* B1;           // optional part 1 (see n_split / k_split)
    int64_t ldb1;
    int64_t b1_seg_stride;
    int n_split;              // rows n >= n_split come from B1 (default: N)
    int k_split;              // columns k >= k_split come from B1 (default: K)
    void* C;                  // output, row stride ldc
    int64_t ldc;
    int c_f32;                // 1: C is float32; 0: C is dtype
    const int32_t* c_rows;    // optional scatter: C row = c_rows[m] / c_div
    int c_div;
    const float* bias;        // optional [N]
    const float* row_scale;   // optional: columns n >= scale_col0 of row m are
    const int32_t* scale_rows;//   scaled by row_scale[scale_rows[m]]
    int scale_col0;
    int gelu;                 // 1: GELU after bias
    int64_t M;                // rows (sum of segments when grouped)
    int N, K;
    const int32_t* seg_offsets;  // optional [nseg+1] on the device: grouped GEMM
    int nseg;
};
// A GemmDesc with the neutral defaults for the optional fields.
inline GemmDesc gemm_desc(int64_t M, int N, int K) {
    GemmDesc g{};
    g.a_div = 1;
    g.c_div = 1;
    g.n_split = N;
    g.k_split = K;
    g.M = M;
    g.N = N;
    g.K = K;
    return g;
}
hipError_t launch_gemm(int dtype, const GemmDesc& g, hipStream_t st);

}  // namespace clearmoe
