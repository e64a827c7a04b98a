// Internal declarations of the CLEAR-MoE HIP kernels (gfx950) and their host
// launchers.  Nothing here is part of the public C ABI (include/clearmoe.h).
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace clearmoe {

// ---------------------------------------------------------------------------
// Kernel launches.  Every kernel goes through launch_kernel, so that a timed
// stage can have its kernel's own start and end written into two events by
// the dispatch itself (hipExtLaunchKernel): no marker packets join the
// stream, and the timed step runs as an untimed one does.
// ---------------------------------------------------------------------------
struct LaunchTiming {
    hipEvent_t start = nullptr, stop = nullptr;   // both set, or both null
};
// The calling thread's pending timing (defined with the stage timer).
LaunchTiming& launch_timing();

// Launch on st; the first launch after a timed stage opens takes its events.
// Errors are left for the caller's hipGetLastError.
template <typename... KArgs, typename... Args>
void launch_kernel(void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t lds, hipStream_t st,
                   Args... args) {
    LaunchTiming& t = launch_timing();
    const LaunchTiming use = t;
    t = LaunchTiming{};
    hipExtLaunchKernelGGL(kernel, grid, block, static_cast<std::uint32_t>(lds), st, use.start,
                          use.stop, 0u, static_cast<KArgs>(args)...);
}

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

// Two floats -> two bf16 by the hardware conversion (round to nearest even),
// packed in 32 bits, first value in the low half.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack2_bf16(float a, float b) {
    const f32x2_t v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}

template <typename T> struct Elem;
template <> struct Elem<float> {
    static constexpr int per16 = 4;                 // elements per 16-byte piece
    __device__ static float load(const float* p, int64_t i) { return p[i]; }
    __device__ static float to_f32(float v) { return v; }
    __device__ static float from_f32(float v) { return v; }
    // four consecutive elements (16-byte aligned)
    __device__ static void store4(float* p, const float (&v)[4]) {
        *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
    }
};
template <> struct Elem<bf16_bits> {
    static constexpr int per16 = 8;
    __device__ static float load(const bf16_bits* p, int64_t i) { return bf16_to_f32(p[i]); }
    __device__ static float to_f32(bf16_bits v) { return bf16_to_f32(v); }
    __device__ static bf16_bits from_f32(float v) { return f32_to_bf16(v); }
    // four consecutive elements (8-byte aligned)
    __device__ static void store4(bf16_bits* p, const float (&v)[4]) {
        uint2 w;
        w.x = pack2_bf16(v[0], v[1]);
        w.y = pack2_bf16(v[2], v[3]);
        *reinterpret_cast<uint2*>(p) = w;
    }
};

// Exact-erf GELU, v Phi(v) = 0.5 v (1 + erf(v / sqrt 2)), in float32.
// erf by Abramowitz & Stegun 7.1.26 (|error| <= 1.5e-7 for every argument):
// for a >= 0, 1 - erf(a) = t P(t) exp(-a^2), t = 1 / (1 + p a), P of degree 4.
// With a = |v| / sqrt 2 and h = 0.5 |v| (1 - erf(a)) >= 0, GELU(v) = v - h for
// v >= 0 and -h for v < 0, i.e. max(v, 0) - h (no cancellation in the
// negative tail).  The 0.5 is folded into P's coefficients and 1 / sqrt 2
// into p, exp(-a^2) = 2^(-v^2 log2(e) / 2), and the reciprocal and power of
// two are the hardware instructions (about 1 ulp): 12 FMA-class operations
// and 2 transcendental ones.
__device__ __forceinline__ float gelu_erf(float v) {
    const float t = __builtin_amdgcn_rcpf(__builtin_fmaf(fabsf(v), 0.23164188827f, 1.0f));   // p / sqrt 2
    float hp = __builtin_fmaf(t, 0.5307027145f, -0.7265760135f);   // 0.5 * (a5, a4)
    hp = __builtin_fmaf(t, hp, 0.7107068705f);                      // 0.5 * a3
    hp = __builtin_fmaf(t, hp, -0.142248368f);                      // 0.5 * a2
    hp = __builtin_fmaf(t, hp, 0.127414796f);                       // 0.5 * a1
    const float e = __builtin_amdgcn_exp2f(v * v * -0.72134752044448170368f);   // -log2(e) / 2
    const float h = fabsf(v) * (t * hp) * e;
    return fmaxf(v, 0.0f) - h;
}

// Raw buffer resources (gfx950): a 16-byte load at an offset outside
// [0, bytes) returns zeros, so tails need neither branches nor a zero page,
// and the loads stay in the vector-memory counter (a select between two
// pointers of different address spaces turns loads into flat ones, which
// also count against the 4-bit LDS/scalar counter and so stall a wave after
// 15 outstanding loads).  bytes must be below 2^31.
constexpr uint32_t kRawOob = 0x80000000u;        // an offset past every resource
constexpr int kRawWord3 = 0x00020000;            // raw dword access

__device__ __forceinline__ __amdgpu_buffer_rsrc_t raw_rsrc(const void* p, int64_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), static_cast<short>(0),
                                             static_cast<int>(bytes), kRawWord3);
}
__device__ __forceinline__ uint4 raw_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<int>(off), 0, 0));
}

// ---------------------------------------------------------------------------
// Tiling constants shared by host and device code.
// ---------------------------------------------------------------------------
constexpr int kRouteTile = 256;      // tokens per dispatch tile (permutation workgroup)
constexpr int kSmallTile = 64;       // tokens per histogram tile for small token counts
// Largest tile histogram (tiles x experts) scanned inline by the permutation.
constexpr int64_t kInlineScanMax = 8192;

__host__ __device__ inline int64_t route_tiles(int64_t T) { return (T + kRouteTile - 1) / kRouteTile; }
// Tokens per histogram tile (the router's workgroup): 64 when there are few
// tokens (E <= 16 and the 64-token histogram still fits the permutation's
// inline scan), so that a small token count spreads over four times as many
// workgroups; otherwise 256.  A function of T and E only: the router and the
// dispatch agree on it.
__host__ __device__ inline int hist_tile(int64_t T, int E) {
    return (E <= 16 && (T + kSmallTile - 1) / kSmallTile * E <= kInlineScanMax) ? kSmallTile : kRouteTile;
}
__host__ __device__ inline int64_t hist_tiles(int64_t T, int E) {
    const int h = hist_tile(T, E);
    return (T + h - 1) / h;
}

// ---------------------------------------------------------------------------
// Host launchers (return hipError_t of the launch).
// ---------------------------------------------------------------------------
// Router logits (float32 MFMA, certified; double recompute of near ties),
// top-k (adaptive != 0: top-1 / top-2 by confidence tau, k = 2 slots), gates,
// per-tile expert histogram (tile_counts may be NULL).  dense_stride > 0:
// tokens t with t % dense_stride == 0 get no expert (all slots -1, gate 0).
hipError_t launch_route(int dtype, const void* x, const void* Wg, const float* bg, int64_t T,
                        int D, int E, int k, int adaptive, int renorm, double tau, int dense_stride,
                        int32_t* idx, float* gate, int32_t* tile_counts, hipStream_t st);
// MLP router: hidden GELU(x Wh^T + bh) of width Hr (1..kMlpHiddenMax) rounded
// to the storage type, logits hr Wo^T + bo in double; then as launch_route
// (no histogram).
hipError_t launch_route_mlp(int dtype, const void* x, const void* Wh, const float* bh,
                            const void* Wo, const float* bo, int64_t T, int D, int Hr, int E,
                            int k, int adaptive, int renorm, double tau, int dense_stride, int32_t* idx,
                            float* gate, hipStream_t st);
constexpr int kMlpHiddenMax = 256;
// Per-tile expert histogram of an index array (tiles of hist_tile(T, E) tokens).
hipError_t launch_tile_histogram(const int32_t* idx, int64_t T, int E, int k,
                                 int32_t* tile_counts, hipStream_t st);
// Chunked exclusive scan of 256-token tile histograms: for tile b in chunk
// c = b / 256, tile_base[b][e] = sum of tile_counts[b'][e] over the earlier
// tiles b' of chunk c, and chunk_tot[c][e] = the chunk's column sums
// (scan_chunks(ntiles) chunks, all scanned in parallel).
int64_t scan_chunks(int64_t ntiles);
hipError_t launch_scan(const int32_t* tile_counts, int64_t ntiles, int E, int32_t* tile_base,
                       int32_t* chunk_tot, hipStream_t st);
// Stable permutation (and optional row copy x -> xperm), one workgroup per
// 256 tokens.  With tile_counts non-NULL the histogram (tiles of
// hist_tile(T, E) tokens) is scanned inline (tile_base unused) and
// counts/offsets are written; otherwise tile_base/offsets come from
// launch_scan over 256-token tiles (tile bases within a chunk, plus the
// chunk totals, from which the permutation forms counts and offsets).  An
// index of -1 is an empty slot: inv = -1, and perm[offsets[E] .. T*k) = -1.
hipError_t launch_permute(int dtype, const int32_t* idx, const int32_t* tile_base,
                          const int32_t* chunk_tot, int32_t* offsets, const int32_t* tile_counts,
                          int32_t* counts, int64_t T, int E, int k, int32_t* perm, int32_t* inv,
                          const void* x, void* xperm, int D, hipStream_t st);
// y[t] = sum_j gate[t,j] ye[inv[t*k+j]]  (ye, y in dtype).
hipError_t launch_combine_gated(int dtype, const void* ye, const int32_t* inv, const float* gate,
                                void* y, int64_t T, int D, int k, hipStream_t st);
// y[t] = hsh[t] + sum_j hres[inv[t*k+j]]  (hsh, hres float32; y in dtype);
// hres has hres_rows rows (other positions count as zero rows).
hipError_t launch_combine_residual(int dtype, const float* hsh, const float* hres,
                                   const int32_t* inv, void* y, int64_t T, int D, int k,
                                   int64_t hres_rows, hipStream_t st);
// Pair order of a top-2 routing (idx, gate [T, 2]): a token with one expert
// e (the other slot empty, as the adaptive router leaves it) gets key e; one
// with experts a < b gets key E + pair_index(a, b), the pairs numbered in
// lexicographic order (pair_index(a, b) = a (2E - a - 1) / 2 + b - a - 1); one
// with none gets -1.  ga[t], gb[t] = the gates of a and b (gate of e and 0
// for one expert).  The E (E + 1) / 2 keys must not exceed kPairMaxKeys.
constexpr int kPairMaxKeys = 64;
__host__ __device__ inline int pair_keys(int E) { return E * (E + 1) / 2; }
// Experts (a, b) of pair number s (0 <= s < E (E - 1) / 2).
__host__ __device__ inline void pair_experts(int s, int E, int& a, int& b) {
    a = 0;
    while (s >= E - 1 - a) {
        s -= E - 1 - a;
        ++a;
    }
    b = a + 1 + s;
}
// Also writes the key histogram of every tile of hist_tile(T, pair_keys(E))
// tokens into tile_counts [hist_tiles(T, pair_keys(E))][pair_keys(E)], as
// the dispatch over keys reads it.
hipError_t launch_pair_key(const int32_t* idx, const float* gate, int64_t T, int E, int32_t* key,
                           float* ga, float* gb, int32_t* tile_counts, hipStream_t st);
// out = x + f (dtype, [T, D], D a multiple of 8 for bf16 / 4 for float32).
hipError_t launch_residual_add(int dtype, const void* x, const void* f, void* out, int64_t T, int D,
                               hipStream_t st);
// dst[b][r][c] = src[b][r][c] for r < srows, c < scols, else 0, over
// b < batches, r < drows, c < dcols (elements of elem_bytes = 2 or 4 bytes;
// src and dst each contiguous).  Pads with zeros (drows >= srows, dcols >=
// scols) or crops (drows <= srows, dcols <= scols).
hipError_t launch_pad_copy(int elem_bytes, const void* src, void* dst, int64_t batches, int64_t srows,
                           int64_t scols, int64_t drows, int64_t dcols, hipStream_t st);
// Any row width D, one element per thread: xperm[p] = x[perm[p] / k] for
// p < *nreal (a device count, e.g. offsets[E]; A = T k rows at most), and
// the gated combine y[t] = sum_j gate[t, j] ye[inv[t k + j]] (as
// launch_combine_gated).
hipError_t launch_gather_rows_elem(int dtype, const void* x, const int32_t* perm,
                                   const int32_t* nreal, int64_t A, int k, int D, void* xperm,
                                   hipStream_t st);
hipError_t launch_combine_gated_elem(int dtype, const void* ye, const int32_t* inv,
                                     const float* gate, void* y, int64_t T, int D, int k,
                                     hipStream_t st);
// Index maps of the padded-batch backend (expert e owns rows [e C, e C + C)):
// perm_pad [E C] (-1 = padding), inv_pad [A], seg [E + 1] = e C.
hipError_t launch_pad_index(const int32_t* idx, const int32_t* counts, const int32_t* offsets,
                            const int32_t* perm, const int32_t* inv, int64_t A, int E, int64_t C,
                            int32_t* perm_pad, int32_t* inv_pad, int32_t* seg, hipStream_t st);

// NT GEMM  C[crow(m), n] = epi( sum_k A[arow(m), k] B_seg(m)[n, k] ).
// B may come in up to three parts: rows n_split <= n < n_split2 from B1 (row
// n - n_split) and rows n >= n_split2 from B2 (row n - n_split2), or columns
// k_split <= k < k_split2 from B1 and k >= k_split2 from B2; each part has
// its own per-segment stride (0 = shared by all segments).  Parts 1 and 2
// take the segment's index, or with pair_E > 0 (segment s = the s-th expert
// pair (a, b), a < b, of a top-2 pair order; see pair_experts) a for B1 and b
// for B2.  With seg_merge the segments' rows form one range, all with the
// parts of segment 0.
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
    const void* B2;           // optional part 2
    int64_t ldb2;
    int64_t b2_seg_stride;
    int n_split;              // rows n >= n_split come from B1 (default: N)
    int n_split2;             // rows n >= n_split2 come from B2 (default: N)
    int k_split;              // columns k >= k_split come from B1 (default: K)
    int k_split2;             // columns k >= k_split2 come from B2 (default: K)
    int pair_E;               // > 0: segments are expert pairs (see above)
    int seg_merge;            // 1: rows [seg_offsets[0], seg_offsets[nseg]) as one segment
    void* C;                  // output, row stride ldc
    int64_t ldc;
    int c_f32;                // 1: C is float32; 0: C is dtype
    const int32_t* c_rows;    // optional scatter: C row = c_rows[m] / c_div
    int c_div;
    const float* bias;        // optional [N]
    const float* row_scale;   // optional: columns scale_col0 <= n < scale_col1 of
    const int32_t* scale_rows;//   row m are scaled by row_scale[scale_rows[m]],
    int scale_col0;           //   columns n >= scale_col1 by row_scale2[...]
    int scale_col1;           //   (a negative scale row scales by 0)
    const float* row_scale2;
    int gelu;                 // 1: GELU after bias
    int64_t M;                // rows (sum of segments when grouped)
    int N, K;
    const int32_t* seg_offsets;  // optional [nseg+1] on the device: grouped GEMM
    int nseg;
    // optional split K for products with few tiles and long K (see
    // gemm_ksplit): float32 partial tiles (kGemmKsplitBytes) and per-tile
    // arrival counters (kGemmKsplitTiles int32) of workspace
    float* ks_part;
    int32_t* ks_count;
};
constexpr size_t kGemmKsplitBytes = static_cast<size_t>(256) * 64 * 128 * 4;
constexpr int kGemmKsplitTiles = 128;
// A GemmDesc with the neutral defaults for the optional fields.
inline GemmDesc gemm_desc(int64_t M, int N, int K) {
    GemmDesc g{};
    g.a_div = 1;
    g.c_div = 1;
    g.n_split = N;
    g.n_split2 = N;
    g.k_split = K;
    g.k_split2 = K;
    g.scale_col1 = N;
    g.M = M;
    g.N = N;
    g.K = K;
    return g;
}
hipError_t launch_gemm(int dtype, const GemmDesc& g, hipStream_t st);

// Fused top-1 layer in bfloat16: y[perm p] = [t|u](p) [US | P_e]^T + b2 with
// [t|u](p) = GELU(x[perm p] W1^T + b1) [Vt ; Q_e]^T (u columns times the gate),
// every intermediate on chip.  Needs the expert order of a top-1 routing:
// either (perm, offsets) from the dispatch, or (tile_counts non-NULL) the
// router's tile histogram and idx, from which each workgroup finds its rows'
// tokens itself (histograms of at most kInlineScanMax entries).  Shapes
// outside fused_top1_supported use the GEMM path.
constexpr int kFusedMaxD = 384;      // six 64-wide input groups; x rows of a 64-row tile live in LDS ...
constexpr int kFusedMaxH = 8192;     // ... beside b1
constexpr int kFusedMaxRQ = 160;     // [t|u] accumulators live in registers
bool fused_top1_supported(int D, int H, int r, int q);
struct ClassArgs;
// With cls (a planned class_ffn pass, class_ffn.h) the class rows' dense FFN
// runs on extra workgroups of the same launch; only for a launch without
// the hidden split (fused_split(T, E, H) == 1), else an invalid-value error.
hipError_t launch_fused_top1(const void* x, const void* W1, const float* b1, const void* US,
                             const void* Vt, const float* b2, const void* P, const void* Q,
                             const int32_t* perm, const int32_t* offsets, const int32_t* idx,
                             const int32_t* tile_counts, const float* gate, void* y, int64_t T,
                             int D, int H, int E, int r, int q, float* part, int32_t* counters,
                             hipStream_t st, const ClassArgs* cls = nullptr);
// Small batches (fewer 64-row tiles than CUs) split each tile's hidden units
// over fused_split(T, E, H) workgroups; the launch then needs part
// (fused_part_bytes) and counters (T / 64 + E + 1 int32) of workspace, else
// both may be NULL.
int fused_split(int64_t T, int E, int H);
size_t fused_part_bytes(int64_t T, int E, int H, int r, int q);

}  // namespace clearmoe
