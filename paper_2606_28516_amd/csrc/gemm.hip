// LDS-tiled MFMA NT GEMM for the CLEAR-MoE layer (gfx950):
//     C[m, n] = epi( sum_k A[arow(m), k] * B_seg(m)[n, k] )
// used for fc1 + GELU (Eq. 2), the two skinny products of the shared SVD basis
// and, grouped by expert with device-resident segment offsets, the two
// products of the per-expert residual (Algorithm 3, one product per
// contiguous expert sub-batch, with no host round trip for the sizes).
//
// Mapping
//   * 256 threads = 4 waves in a WM x WN grid; a wave owns a (BM/WM) x (BN/WN)
//     block of 32x32 MFMA tiles with float32 accumulators;
//   * bf16: v_mfma_f32_32x32x16_bf16, each lane feeds 8 consecutive k of one
//     row (A) / one column (B);  f32: v_mfma_f32_32x32x2f32, each lane holds 4
//     consecutive k per operand and the two lane halves take k and k+4 in
//     four successive MFMAs (the k order of a dot product is free, and A and B
//     use the same order);
//   * per stage each row contributes 128 bytes of k; LDS rows are padded to
//     144 bytes, so the 16-byte reads of 32 consecutive rows are conflict free;
//   * global -> register -> LDS double buffering: the next stage's 16-byte
//     loads are in flight while the current stage feeds the MFMAs.
//   * grouped mode: workgroup x-index enumerates (segment, M-tile) pairs in
//     segment order, read from the device offsets; surplus workgroups exit.
#include "kernels.h"

namespace clearmoe {

constexpr int kGemmStageBytes = 128;             // bytes of k per row per stage
constexpr int kGemmLdsStride = kGemmStageBytes + 16;

template <typename Tin> struct Mfma;
template <> struct Mfma<bf16_bits> {
    __device__ static void step(const uint4& a, const uint4& b, f32x16& c) {
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                     __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }
};
template <> struct Mfma<float> {
    __device__ static void step(const uint4& a, const uint4& b, f32x16& c) {
        const f32x4 av = __builtin_bit_cast(f32x4, a);
        const f32x4 bv = __builtin_bit_cast(f32x4, b);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(av[0], bv[0], c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(av[1], bv[1], c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(av[2], bv[2], c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_32x32x2f32(av[3], bv[3], c, 0, 0, 0);
    }
};

template <typename Tin, int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(256) void k_gemm(GemmDesc g) {
    static_assert(WM * WN == 4, "4 waves");
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 32, TN = WTN / 32;
    static_assert(TM >= 1 && TN >= 1, "wave tile at least 32x32");
    constexpr int PER16 = Elem<Tin>::per16;
    constexpr int BK = kGemmStageBytes / static_cast<int>(sizeof(Tin));  // elements per stage
    constexpr int PIECES = kGemmStageBytes / 16;                          // 16B pieces per row
    constexpr int ALOADS = BM * PIECES / 256;
    constexpr int BLOADS = (BN * PIECES + 255) / 256;
    __shared__ __align__(16) unsigned char sA[2][BM * kGemmLdsStride];
    __shared__ __align__(16) unsigned char sB[2][BN * kGemmLdsStride];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;

    // ---- which rows (and which expert segment) this workgroup owns
    int64_t m_lo, m_hi;
    int seg = 0;
    if (g.seg_offsets != nullptr) {
        const int64_t bid = blockIdx.x;
        int64_t before = 0;
        bool found = false;
        for (int e = 0; e < g.nseg; ++e) {
            // offsets are clamped to [0, M] so a bad offsets array cannot send a
            // workgroup outside the buffers
            int64_t lo = g.seg_offsets[e], hi = g.seg_offsets[e + 1];
            lo = lo < 0 ? 0 : (lo > g.M ? g.M : lo);
            hi = hi < lo ? lo : (hi > g.M ? g.M : hi);
            const int64_t nt = (hi - lo + BM - 1) / BM;
            if (bid < before + nt) {
                seg = e;
                m_lo = lo + (bid - before) * BM;
                m_hi = m_lo + BM < hi ? m_lo + BM : hi;
                found = true;
                break;
            }
            before += nt;
        }
        if (!found) return;                      // uniform over the workgroup
    } else {
        m_lo = static_cast<int64_t>(blockIdx.x) * BM;
        if (m_lo >= g.M) return;
        m_hi = m_lo + BM < g.M ? m_lo + BM : g.M;
    }
    const int n0 = blockIdx.y * BN;
    const Tin* A = static_cast<const Tin*>(g.A);
    const Tin* B = static_cast<const Tin*>(g.B) + static_cast<int64_t>(seg) * g.b_seg_stride;

    // ---- per-thread source rows of the global loads
    int64_t arow[ALOADS];
#pragma unroll
    for (int i = 0; i < ALOADS; ++i) {
        const int r = (tid + i * 256) / PIECES;
        const int64_t m = m_lo + r;
        int64_t src = -1;
        if (m < m_hi) src = g.a_rows != nullptr ? static_cast<int64_t>(g.a_rows[m] / g.a_div) : m;
        arow[i] = src;
    }

    uint4 ra[ALOADS], rb[BLOADS];
    auto gload = [&](int kt) {
        const int kbase = kt * BK;
#pragma unroll
        for (int i = 0; i < ALOADS; ++i) {
            const int pc = (tid + i * 256) % PIECES;
            const int kk = kbase + pc * PER16;
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (arow[i] >= 0 && kk < g.K)
                v = *reinterpret_cast<const uint4*>(A + arow[i] * g.lda + kk);
            ra[i] = v;
        }
#pragma unroll
        for (int i = 0; i < BLOADS; ++i) {
            const int piece = tid + i * 256;
            const int r = piece / PIECES, pc = piece % PIECES;
            const int kk = kbase + pc * PER16;
            const int n = n0 + r;
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (r < BN && n < g.N && kk < g.K)
                v = *reinterpret_cast<const uint4*>(B + static_cast<int64_t>(n) * g.ldb + kk);
            rb[i] = v;
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < ALOADS; ++i) {
            const int piece = tid + i * 256;
            const int r = piece / PIECES, pc = piece % PIECES;
            *reinterpret_cast<uint4*>(&sA[buf][r * kGemmLdsStride + pc * 16]) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < BLOADS; ++i) {
            const int piece = tid + i * 256;
            const int r = piece / PIECES, pc = piece % PIECES;
            if (r < BN) *reinterpret_cast<uint4*>(&sB[buf][r * kGemmLdsStride + pc * 16]) = rb[i];
        }
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

    const int nk = (g.K + BK - 1) / BK;
    if (nk > 0) {
        gload(0);
        lstore(0);
        __syncthreads();
    }
    const int lrow = lane & 31, lhalf = lane >> 5;
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
        for (int s = 0; s < kGemmStageBytes / 32; ++s) {
            uint4 fa[TM], fb[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                fa[i] = *reinterpret_cast<const uint4*>(
                    &sA[buf][(wm * WTM + i * 32 + lrow) * kGemmLdsStride + s * 32 + lhalf * 16]);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                fb[j] = *reinterpret_cast<const uint4*>(
                    &sB[buf][(wn * WTN + j * 32 + lrow) * kGemmLdsStride + s * 32 + lhalf * 16]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) Mfma<Tin>::step(fa[i], fb[j], acc[i][j]);
        }
        if (kt + 1 < nk) lstore(buf ^ 1);
        __syncthreads();
    }

    // ---- epilogue: D[v] of a 32x32 tile sits at row 8*(v/4) + 4*(lane/32) + v%4, column lane%32
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int n = n0 + wn * WTN + j * 32 + lrow;
            const float bn = (g.bias != nullptr && n < g.N) ? g.bias[n] : 0.0f;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t m = m_lo + wm * WTM + i * 32 + 8 * (v >> 2) + 4 * lhalf + (v & 3);
                if (m >= m_hi || n >= g.N) continue;
                float val = acc[i][j][v];
                if (g.row_scale != nullptr) val *= g.row_scale[g.scale_rows[m]];
                val += bn;
                if (g.gelu) val = gelu_erf(val);
                if (g.c_f32)
                    static_cast<float*>(g.C)[m * g.ldc + n] = val;
                else
                    static_cast<Tin*>(g.C)[m * g.ldc + n] = Elem<Tin>::from_f32(val);
            }
        }
    }
}

template <typename Tin, int BM, int BN, int WM, int WN>
static hipError_t gemm_cfg(const GemmDesc& g, hipStream_t st) {
    int64_t mt = (g.M + BM - 1) / BM;
    if (g.seg_offsets != nullptr) mt += g.nseg;
    const int nt = (g.N + BN - 1) / BN;
    if (mt == 0 || nt == 0) return hipSuccess;
    k_gemm<Tin, BM, BN, WM, WN><<<dim3(static_cast<unsigned>(mt), nt), 256, 0, st>>>(g);
    return hipGetLastError();
}

template <typename Tin>
static hipError_t gemm_dt(const GemmDesc& g, hipStream_t st) {
    if (g.N <= 32) return gemm_cfg<Tin, 128, 32, 4, 1>(g, st);
    if (g.N <= 64) return gemm_cfg<Tin, 128, 64, 4, 1>(g, st);
    return gemm_cfg<Tin, 128, 128, 2, 2>(g, st);
}

hipError_t launch_gemm(int dtype, const GemmDesc& g, hipStream_t st) {
    if (dtype == 0) return gemm_dt<float>(g, st);
    return gemm_dt<bf16_bits>(g, st);
}

}  // namespace clearmoe
