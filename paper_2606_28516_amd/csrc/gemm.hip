// LDS-tiled MFMA NT GEMM for the CLEAR-MoE layer (gfx950):
//     C[m, n] = epi( sum_k A[arow(m), k] * B_seg(m)[n, k] )
// used for fc1 + GELU (Eq. 2), the two skinny products of the shared SVD basis
// and, grouped by expert with device-resident segment offsets, the two
// products of the per-expert residual (Algorithm 3: one product per
// contiguous expert sub-batch, here with no host round trip for the sizes).
//
// Mapping
//   * 4 or 8 waves in a WM x WN grid; a wave owns a (BM/WM) x (BN/WN)
//     block of 32x32 MFMA tiles with float32 accumulators;
//   * bf16: v_mfma_f32_32x32x16_bf16, a lane feeds 8 consecutive k of one row
//     (A) / one column (B); f32: v_mfma_f32_32x32x2f32, a lane holds 4
//     consecutive k per operand and the two lane halves take k and k+4 in four
//     successive MFMAs (the k order of a dot product is free and A and B use
//     the same order);
//   * operands move HBM -> LDS with gfx950's global_load_lds_dwordx4 (no
//     register staging): a stage is 128 bytes of k per row, rows are stored
//     unpadded with the 16-byte chunk index XOR-swizzled by (row >> 1) & 7.
//     A 128-bit LDS read serves 16 lanes per cycle across 64 banks (256 bytes),
//     and the 16 lanes of a group read one chunk of 16 consecutive rows: row
//     parity picks the bank half and the swizzle spreads the 8 rows of each
//     parity over the 8 chunk slots, so the reads are conflict free (a plain
//     row & 7 swizzle puts rows r and r + 8 on the same banks);
//   * NS stages are in flight: stage kt+NS-1 is issued while stage kt feeds
//     the MFMAs, and each wave waits with an explicit vmcnt for exactly its
//     own loads of stage kt before the workgroup barrier;
//   * lanes whose row or k chunk is outside the operand load a 16-byte zero
//     page instead, so tails need no special path and never read out of bounds;
//   * tiles are spread by row tile over the XCDs: workgroup i runs on XCD
//     i % 8, which takes every eighth row tile, in groups of four row tiles
//     whose column tiles it runs column by column, so the A rows and the B
//     rows that the concurrent workgroups of an XCD read are shared among
//     them in its L2, and the leading row tiles (all a grouped product's rows
//     when its segments hold few) use every XCD;
//   * long-K products stage each wave's output rows through LDS and store
//     whole rows (16 bytes per lane) instead of 8-byte pieces;
//   * grouped mode: the tile index enumerates (segment, M-tile) pairs in
//     segment order, read from the device offsets; surplus workgroups exit.
#include "kernels.h"

namespace clearmoe {

constexpr int kStageBytes = 128;   // bytes of k per row per stage (default)
constexpr int kXcds = 8;           // MI355X: 8 XCDs of 32 CUs

__device__ __attribute__((aligned(16))) const uint32_t g_zero_page[4] = {0u, 0u, 0u, 0u};

typedef __attribute__((address_space(3))) uint32_t lds_u32;

// Physical 16-byte chunk slot of logical chunk c in LDS row r is c ^ swz(r),
// for rows of SB bytes (CPR = SB / 16 chunks): a 256-byte bank window holds
// 16 / CPR rows, and the swizzle spreads the CPR rows that share window
// positions over the CPR chunk slots, so 16 consecutive rows of one logical
// chunk hit 16 distinct 16-byte bank groups.
template <int SB>
__device__ __forceinline__ int swz(int r) {
    constexpr int CPR = SB / 16, RW = 16 / CPR;
    return (r / RW) % CPR;
}

// 16 bytes per lane, HBM -> LDS: lane i's bytes land at lds_base + 16*i.
// Issued as inline asm so that the compiler does not model it: the waits for
// these loads are the explicit per-wave vmcnt waits plus the workgroup barrier
// of the pipeline below.  M0 holds the LDS base; one wait state is required
// between writing M0 and the load that reads it.
__device__ __forceinline__ void async_load16(const void* gptr, uint32_t lds_base) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                 :
                 : "s"(lds_base), "v"(gptr)
                 : "memory", "m0");
}

// s_waitcnt vmcnt(n) (gfx9 encoding), other counters untouched.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

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

// WPE > 0 asks for WPE waves per SIMD (registers capped to fit them).
template <typename Tin, int BM, int BN, int WM, int WN, int NS, int SB = kStageBytes, int WPE = 0>
__global__ __launch_bounds__(64 * WM * WN) __attribute__((amdgpu_waves_per_eu(WPE > 0 ? WPE : 1)))
void k_gemm(GemmDesc g, int mtiles, int ntiles, int group, int ksplit, int staged) {
    constexpr int NW = WM * WN;                     // waves: 4 (one per SIMD) or 8 (two)
    static_assert(NW == 4 || NW == 8, "4 or 8 waves");
    constexpr int WTM = BM / WM, WTN = BN / WN;
    constexpr int TM = WTM / 32, TN = WTN / 32;
    static_assert(TM >= 1 && TN >= 1, "wave tile at least 32x32");
    static_assert(SB == 64 || SB == 128, "stage rows of 64 or 128 bytes");
    constexpr int CPR = SB / 16;                    // 16-byte chunks per stage row
    constexpr int RPL = 64 / CPR;                   // rows per load instruction (1 KB)
    static_assert(BM % (RPL * NW) == 0 && BN % (RPL * NW) == 0, "whole load groups per wave");
    constexpr int PER16 = Elem<Tin>::per16;
    constexpr int BK = SB / static_cast<int>(sizeof(Tin));
    constexpr int AL = BM / (RPL * NW), BL = BN / (RPL * NW);   // load instructions per wave per stage
    constexpr int LPS = AL + BL;
    static_assert(LPS * (NS - 1) < 64, "vmcnt range");
    constexpr int STAGE_A = BM * SB, STAGE_B = BN * SB;
    // One LDS array per stage, so that with the stage index a compile-time
    // constant the LDS lowering gives each its own alias scope and the
    // compiler's own waits for the async loads cover only the stage read.
    __shared__ __attribute__((aligned(1024))) unsigned char st0[STAGE_A + STAGE_B];
    __shared__ __attribute__((aligned(1024))) unsigned char st1[NS > 1 ? STAGE_A + STAGE_B : 16];
    __shared__ __attribute__((aligned(1024))) unsigned char st2[NS > 2 ? STAGE_A + STAGE_B : 16];
    __shared__ __attribute__((aligned(1024))) unsigned char st3[NS > 3 ? STAGE_A + STAGE_B : 16];
    static_assert(NS >= 2 && NS <= 4, "2..4 stages");

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;

    // ---- tile of this workgroup.  Workgroup b runs on XCD x = b % 8 as its
    //      i-th (i = b / 8); XCD x owns the row tiles x, x + 8, x + 16, ...
    //      (mx of them) and takes them in groups of `group` row tiles (the
    //      last group may be short), each group column tile by column tile,
    //      so the workgroups in flight on one XCD share both their A rows and
    //      their B rows in its L2, and the first row tiles -- the only ones
    //      with rows when a grouped product's segments hold fewer rows than
    //      its bound M -- spread over every XCD.  With split K, S consecutive
    //      workgroups of one XCD share a tile, part kp taking its share of
    //      the k stages.
    const int S = g.ks_part != nullptr ? ksplit : 1;
    const int xcd = blockIdx.x % kXcds, local = blockIdx.x / kXcds;
    const int tile_local = local / S, kp = local - tile_local * S;
    const int mx = (mtiles - xcd + kXcds - 1) / kXcds;
    const int full = mx / group;
    int mi, nt;
    if (tile_local < full * group * ntiles) {
        const int gi = tile_local / (group * ntiles), r = tile_local - gi * group * ntiles;
        mi = gi * group + r % group;
        nt = r / group;
    } else {
        const int r = tile_local - full * group * ntiles, gm = mx - full * group;
        if (gm <= 0 || r >= gm * ntiles) return;
        mi = full * group + r % gm;
        nt = r / gm;
    }
    const int mt = mi * kXcds + xcd;
    if (mt >= mtiles) return;
    const int tile = mt * ntiles + nt;
    int64_t m_lo, m_hi;
    int seg = 0;
    if (g.seg_offsets != nullptr && g.seg_merge) {
        int64_t lo = g.seg_offsets[0], hi = g.seg_offsets[g.nseg];
        lo = lo < 0 ? 0 : (lo > g.M ? g.M : lo);
        hi = hi < lo ? lo : (hi > g.M ? g.M : hi);
        m_lo = lo + static_cast<int64_t>(mt) * BM;
        if (m_lo >= hi) return;
        m_hi = m_lo + BM < hi ? m_lo + BM : hi;
    } else if (g.seg_offsets != nullptr) {
        int64_t before = 0;
        bool found = false;
        for (int e = 0; e < g.nseg; ++e) {
            // offsets are clamped to [0, M] so a bad offsets array cannot send a
            // workgroup outside the buffers
            int64_t lo = g.seg_offsets[e], hi = g.seg_offsets[e + 1];
            lo = lo < 0 ? 0 : (lo > g.M ? g.M : lo);
            hi = hi < lo ? lo : (hi > g.M ? g.M : hi);
            const int64_t n_t = (hi - lo + BM - 1) / BM;
            if (mt < before + n_t) {
                seg = e;
                m_lo = lo + (mt - before) * BM;
                m_hi = m_lo + BM < hi ? m_lo + BM : hi;
                found = true;
                break;
            }
            before += n_t;
        }
        if (!found) return;                      // uniform over the workgroup
    } else {
        m_lo = static_cast<int64_t>(mt) * BM;
        if (m_lo >= g.M) return;
        m_hi = m_lo + BM < g.M ? m_lo + BM : g.M;
    }
    const int n0 = nt * BN;
    const Tin* A = static_cast<const Tin*>(g.A);
    const Tin* B0 = g.B != nullptr
                        ? static_cast<const Tin*>(g.B) + static_cast<int64_t>(seg) * g.b_seg_stride
                        : nullptr;
    // parts 1 and 2 belong to the segment's expert, or, for pair segments
    // (s = a * pair_E + b), to its experts a and b
    int e1 = seg, e2 = seg;
    if (g.pair_E > 0) pair_experts(seg, g.pair_E, e1, e2);
    const Tin* B1 = g.B1 != nullptr
                        ? static_cast<const Tin*>(g.B1) + static_cast<int64_t>(e1) * g.b1_seg_stride
                        : nullptr;
    const Tin* B2 = g.B2 != nullptr
                        ? static_cast<const Tin*>(g.B2) + static_cast<int64_t>(e2) * g.b2_seg_stride
                        : nullptr;
    const uint32_t* zero = g_zero_page;

    // ---- per-lane source rows of its load instructions (row within the tile
    //      = (wave*AL + i)*8 + lane/8; LDS chunk lane%8 holds global chunk
    //      (lane%8) ^ swz(row)).  A B row has a pointer per k part (the k
    //      split picks between them per chunk).
    const int lrow8 = lane / CPR, cpos = lane % CPR;
    const Tin* arow[AL];
    const Tin* brow0[BL];
    const Tin* brow1[BL];
    const Tin* brow2[BL];
    int achunk[AL], bchunk[BL];
#pragma unroll
    for (int i = 0; i < AL; ++i) {
        const int r = (wave * AL + i) * RPL + lrow8;
        const int64_t m = m_lo + r;
        arow[i] = nullptr;
        if (m < m_hi) {
            // a negative gather index is a padding row: it reads zeros
            const int64_t src = g.a_rows != nullptr ? static_cast<int64_t>(g.a_rows[m]) : m;
            if (src >= 0) arow[i] = A + (g.a_rows != nullptr ? src / g.a_div : src) * g.lda;
        }
        achunk[i] = cpos ^ swz<SB>(r);
    }
#pragma unroll
    for (int i = 0; i < BL; ++i) {
        const int r = (wave * BL + i) * RPL + lrow8;
        const int n = n0 + r;
        brow0[i] = brow1[i] = brow2[i] = nullptr;
        if (n < g.N) {
            if (n < g.n_split) {
                if (g.B != nullptr) brow0[i] = B0 + static_cast<int64_t>(n) * g.ldb;
                if (B1 != nullptr) brow1[i] = B1 + static_cast<int64_t>(n) * g.ldb1;
                if (B2 != nullptr) brow2[i] = B2 + static_cast<int64_t>(n) * g.ldb2;
            } else if (n < g.n_split2) {
                if (B1 != nullptr) brow0[i] = B1 + static_cast<int64_t>(n - g.n_split) * g.ldb1;
            } else if (B2 != nullptr) {
                brow0[i] = B2 + static_cast<int64_t>(n - g.n_split2) * g.ldb2;
            }
        }
        bchunk[i] = cpos ^ swz<SB>(r);
    }

    // k stages of this part: [kb0, kb0 + nk)
    const int nk_all = (g.K + BK - 1) / BK;
    const int kb0 = static_cast<int>(static_cast<int64_t>(kp) * nk_all / S);
    const int nk = static_cast<int>(static_cast<int64_t>(kp + 1) * nk_all / S) - kb0;

    auto stage = [&](int b) -> unsigned char* {
        return b == 0 ? st0 : b == 1 ? st1 : b == 2 ? st2 : st3;
    };

    // Issue the async loads of stage kt into LDS buffer `b` (compile-time).
    auto issue = [&](int kt, int b) {
        const uint32_t base = __builtin_amdgcn_readfirstlane(
            static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_u32*)(stage(b)))));
        const int kbase = (kb0 + kt) * BK;
#pragma unroll
        for (int i = 0; i < AL; ++i) {
            const int kk = kbase + achunk[i] * PER16;
            const void* src = (arow[i] != nullptr && kk < g.K) ? static_cast<const void*>(arow[i] + kk)
                                                               : static_cast<const void*>(zero);
            async_load16(src, __builtin_amdgcn_readfirstlane(base + (wave * AL + i) * 1024));
        }
#pragma unroll
        for (int i = 0; i < BL; ++i) {
            const int kk = kbase + bchunk[i] * PER16;
            const void* src = zero;
            if (kk < g.K) {
                if (kk < g.k_split) {
                    if (brow0[i] != nullptr) src = brow0[i] + kk;
                } else if (kk < g.k_split2) {
                    if (brow1[i] != nullptr) src = brow1[i] + (kk - g.k_split);
                } else if (brow2[i] != nullptr) {
                    src = brow2[i] + (kk - g.k_split2);
                }
            }
            async_load16(src,
                         __builtin_amdgcn_readfirstlane(base + STAGE_A + (wave * BL + i) * 1024));
        }
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

#pragma unroll
    for (int s = 0; s < NS - 1; ++s)
        if (s < nk) issue(s, s);

    const int lrow = lane & 31, lhalf = lane >> 5;
    for (int k0 = 0; k0 < nk; k0 += NS) {
#pragma unroll
        for (int b = 0; b < NS; ++b) {
            const int kt = k0 + b;
            if (kt >= nk) break;
            // this wave's loads of stage kt are done once at most the later
            // stages' loads are outstanding
            const int later = nk - 1 - kt < NS - 2 ? nk - 1 - kt : NS - 2;
            if (later >= 2 && NS >= 4) wait_vmcnt<(NS >= 4 ? 2 * LPS : 0)>();
            else if (later == 1 && NS >= 3) wait_vmcnt<(NS >= 3 ? LPS : 0)>();
            else wait_vmcnt<0>();
            // Bare barrier: __syncthreads() would also drain the later stages'
            // loads (its fence waits for vmcnt 0).  lgkmcnt(0) first, so every
            // wave's LDS reads of the buffer recycled below have completed.
            __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0) only
            __builtin_amdgcn_s_barrier();
            if (kt + NS - 1 < nk) issue(kt + NS - 1, (b + NS - 1) % NS);
            const unsigned char* sa = stage(b);
            const unsigned char* sb = sa + STAGE_A;
#pragma unroll
            for (int s = 0; s < SB / 32; ++s) {
                const int c = 2 * s + lhalf;        // 16-byte chunk of k within the stage
                uint4 fa[TM], fb[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i) {
                    const int r = wm * WTM + i * 32 + lrow;
                    fa[i] = *reinterpret_cast<const uint4*>(sa + r * SB + ((c ^ swz<SB>(r)) << 4));
                }
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const int r = wn * WTN + j * 32 + lrow;
                    fb[j] = *reinterpret_cast<const uint4*>(sb + r * SB + ((c ^ swz<SB>(r)) << 4));
                }
                // B first: tile (i, j) accumulates C^T (see the epilogue)
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j) Mfma<Tin>::step(fb[j], fa[i], acc[i][j]);
            }
        }
    }

    // ---- split K: each part stores its accumulators (float32, 16 per lane
    //      and tile contiguous) with device-scope accesses, waits for them,
    //      and counts itself in; the last part of the tile to arrive sums the
    //      S parts in part order (the same bits whichever part is last) and
    //      runs the epilogue.  The parts of a tile share an XCD.
    if (S > 1) {
        constexpr int kDevScope = 16;   // cache-policy bits: sc1
        constexpr int kTiles = TM * TN;
        const __amdgpu_buffer_rsrc_t rp = raw_rsrc(
            g.ks_part + static_cast<int64_t>(tile) * S * BM * BN, static_cast<int64_t>(S) * BM * BN * 4);
        auto off = [&](int pp, int i, int j, int q) {
            return static_cast<int>(((((pp * NW + wave) * kTiles + i * TN + j) * 64 + lane) * 4 + q) * 16);
        };
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const f32x4 v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                     acc[i][j][4 * q + 3]};
                    __builtin_amdgcn_raw_buffer_store_b128(v, rp, off(kp, i, j, q), 0, kDevScope);
                }
        // release: every wave's partial stores have completed (vmcnt) and the
        // barrier orders them before thread 0's agent-scope release add; the
        // part that sees the count complete acquires at agent scope before
        // any wave reads the partials
        wait_vmcnt<0>();
        __syncthreads();
        __shared__ int s_last;
        if (tid == 0)
            s_last = __hip_atomic_fetch_add(g.ks_count + tile, 1, __ATOMIC_ACQ_REL,
                                            __HIP_MEMORY_SCOPE_AGENT) == S - 1;
        __syncthreads();
        if (!s_last) return;
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    f32x4 sum = __builtin_amdgcn_raw_buffer_load_b128(rp, off(0, i, j, q), 0, kDevScope);
                    for (int pp = 1; pp < S; ++pp) {
                        const f32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rp, off(pp, i, j, q), 0,
                                                                               kDevScope);
                        sum += v;
                    }
#pragma unroll
                    for (int t = 0; t < 4; ++t) acc[i][j][4 * q + t] = sum[t];
                }
    }

    // ---- staged epilogue (2-byte outputs, N and ldc multiples of 8): each
    //      wave writes a 32-row block of its tile, rounded, to its own slot of
    //      the stage buffers (rows padded by 8 bytes, so the 32 rows of one
    //      8-byte write start on distinct bank pairs), then reads it back as
    //      whole rows, WTN / 8 lanes per row with 16 bytes each, and stores
    //      them; the row scatter applies per stored row.  Same values and
    //      rounding as the direct epilogue below.
    constexpr int kPitch = WTN * 2 + 8;
    constexpr bool kStaged = sizeof(Tin) == 2 && WTN % 8 == 0 && 64 % (WTN / 8) == 0 &&
                             32 % (64 / (WTN / 8)) == 0 && (NW / 2) * 32 * kPitch <= STAGE_A + STAGE_B;
    if (kStaged && staged && !g.c_f32 && g.N % 8 == 0 && g.ldc % 8 == 0) {
        __syncthreads();                   // every wave is done with the stage buffers
        unsigned char* slot = (wave < NW / 2 ? st0 : st1) + (wave % (NW / 2)) * 32 * kPitch;
        constexpr int LPR = WTN / 8, RPI = 64 / LPR;      // lanes per row, rows per read
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int64_t m = m_lo + wm * WTM + i * 32 + lrow;
            float rs = 1.0f, rs1 = 1.0f;
            if (g.row_scale != nullptr && m < m_hi) {
                const int32_t sr = g.scale_rows[m];
                rs = sr >= 0 ? g.row_scale[sr] : 0.0f;
                rs1 = g.row_scale2 == nullptr ? rs : (sr >= 0 ? g.row_scale2[sr] : 0.0f);
            }
#pragma unroll
            for (int j = 0; j < TN; ++j) {
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    const int nl = j * 32 + 8 * q4 + 4 * lhalf;
                    const int n = n0 + wn * WTN + nl;
                    float val[4];
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        const float bb = (g.bias != nullptr && n + t < g.N) ? g.bias[n + t] : 0.0f;
                        const float sc = n + t >= g.scale_col0 ? (n + t >= g.scale_col1 ? rs1 : rs) : 1.0f;
                        val[t] = acc[i][j][4 * q4 + t] * sc + bb;
                        if (g.gelu) val[t] = gelu_erf(val[t]);
                    }
                    uint2 w;
                    w.x = pack2_bf16(val[0], val[1]);
                    w.y = pack2_bf16(val[2], val[3]);
                    *reinterpret_cast<uint2*>(slot + lrow * kPitch + nl * 2) = w;
                }
            }
            // the slot is the wave's own: LDS accesses of one wave complete
            // in order, so only the compiler must keep them in place
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int it = 0; it < 32 / RPI; ++it) {
                const int rr = it * RPI + lane / LPR, ch = lane % LPR;
                const uint4 v = *reinterpret_cast<const uint4*>(slot + rr * kPitch + ch * 16);
                const int64_t mm = m_lo + wm * WTM + i * 32 + rr;
                const int n = n0 + wn * WTN + ch * 8;
                if (mm < m_hi && n < g.N) {
                    const int64_t cr = g.c_rows != nullptr ? static_cast<int64_t>(g.c_rows[mm]) : mm;
                    if (cr >= 0) {
                        const int64_t cm = g.c_rows != nullptr ? cr / g.c_div : cr;
                        *reinterpret_cast<uint4*>(static_cast<Tin*>(g.C) + cm * g.ldc + n) = v;
                    }
                }
            }
            __builtin_amdgcn_wave_barrier();
        }
        return;
    }

    // ---- epilogue.  The MFMAs took B as the first operand, so tile (i, j)
    //      holds C^T: lane l owns row m = .. + i*32 + l%32, and its value v is
    //      column n = .. + j*32 + 8*(v/4) + 4*(l/32) + v%4 -- four consecutive
    //      columns per v-group, written as one 8-byte (bf16) or 16-byte
    //      (float32) store at a row address formed once per tile row.  N is
    //      a multiple of 4 (the shape checks), so a group is all in or all out.
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int64_t m = m_lo + wm * WTM + i * 32 + lrow;
        if (m >= m_hi) continue;
        const int32_t sr = g.row_scale != nullptr ? g.scale_rows[m] : 0;
        float rs = 1.0f, rs1 = 1.0f;
        if (g.row_scale != nullptr) {
            rs = sr >= 0 ? g.row_scale[sr] : 0.0f;
            rs1 = g.row_scale2 == nullptr ? rs : (sr >= 0 ? g.row_scale2[sr] : 0.0f);
        }
        // a negative scatter index is a padding row: it is not stored
        const int64_t cr = g.c_rows != nullptr ? static_cast<int64_t>(g.c_rows[m]) : m;
        if (cr < 0) continue;
        const int64_t cm = g.c_rows != nullptr ? cr / g.c_div : cr;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
#pragma unroll
            for (int q4 = 0; q4 < 4; ++q4) {
                const int n = n0 + wn * WTN + j * 32 + 8 * q4 + 4 * lhalf;
                if (n >= g.N) continue;
                float bb[4] = {0.0f, 0.0f, 0.0f, 0.0f};   // the bias is only 4-byte aligned
                if (g.bias != nullptr) {
#pragma unroll
                    for (int t = 0; t < 4; ++t) bb[t] = g.bias[n + t];
                }
                float val[4];
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const float sc = n + t >= g.scale_col0 ? (n + t >= g.scale_col1 ? rs1 : rs) : 1.0f;
                    val[t] = acc[i][j][4 * q4 + t] * sc + bb[t];
                    if (g.gelu) val[t] = gelu_erf(val[t]);
                }
                if (g.c_f32) {
                    *reinterpret_cast<float4*>(static_cast<float*>(g.C) + cm * g.ldc + n) =
                        make_float4(val[0], val[1], val[2], val[3]);
                } else {
                    Elem<Tin>::store4(static_cast<Tin*>(g.C) + cm * g.ldc + n, val);
                }
            }
        }
    }
}

__global__ void k_zero_tiles(int32_t* c, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) c[i] = 0;
}

// Split K (S parts of every tile's k stages) when the tiles alone would leave
// most CUs idle and every part still has four stages or more.
int gemm_ksplit(int64_t tiles, int nk) {
    if (tiles >= kGemmKsplitTiles || nk < 8) return 1;
    int64_t s = 8;
    if (256 / tiles < s) s = 256 / tiles;
    if (nk / 4 < s) s = nk / 4;
    return s < 2 ? 1 : static_cast<int>(s);
}

template <typename Tin, int BM, int BN, int WM, int WN, int NS, int SB = kStageBytes, int WPE = 0>
static hipError_t gemm_cfg(const GemmDesc& g, hipStream_t st) {
    int64_t mt = (g.M + BM - 1) / BM;
    if (g.seg_offsets != nullptr) mt += g.nseg;
    const int64_t nt = (g.N + BN - 1) / BN;
    const int64_t tiles = mt * nt;
    if (tiles == 0) return hipSuccess;
    constexpr int BK = SB / static_cast<int>(sizeof(Tin));
    // tiles x S <= 256 parts of BM x BN floats each fit kGemmKsplitBytes up
    // to 64 x 128 tiles (larger ones never have so few tiles here)
    int S = 1;
    if (g.ks_part != nullptr && g.ks_count != nullptr && BM * BN <= 64 * 128)
        S = gemm_ksplit(tiles, (g.K + BK - 1) / BK);
    GemmDesc d = g;
    if (S == 1) d.ks_part = nullptr;
    // every XCD takes ceil(mt / 8) row tiles of nt tiles of S parts
    const int64_t per_xcd = (mt + kXcds - 1) / kXcds * nt * S;
    // measured on the DeiT-Base products: groups of four row tiles (fc1 +
    // GELU 391 -> 377 us, the others unchanged); the staged epilogue pays
    // off for long K (dense fc2 298 -> 288, pair [t|u] product 183 -> 178 us)
    // and costs for short K (fc1 +1 %, DeiT-Small fc1 +5 %)
    const int group = 4, staged = g.K >= 2048 ? 1 : 0;
    const int64_t grid = per_xcd * kXcds;
    if (S > 1) {
        // the fill kernel must not take the timing events meant for the GEMM
        LaunchTiming& lt = launch_timing();
        const LaunchTiming keep = lt;
        lt = LaunchTiming{};
        launch_kernel(k_zero_tiles, dim3(1), kGemmKsplitTiles, 0, st, d.ks_count,
                      static_cast<int>(tiles));
        lt = keep;
        const hipError_t err = hipGetLastError();
        if (err != hipSuccess) return err;
    }
    launch_kernel(k_gemm<Tin, BM, BN, WM, WN, NS, SB, WPE>, dim3(static_cast<unsigned>(grid)), 64 * WM * WN, 0, st,
        d, static_cast<int>(mt), static_cast<int>(nt), group, S, staged);
    return hipGetLastError();
}

// Tile choice by shape (measured on MI355X at the layer's sizes): with few
// 128x128 tiles the GEMM is latency bound, so 64-row tiles (more workgroups
// per CU) win; long-K skinny products want 64x64 with four stages in flight;
// the large bfloat16 products take 256x128 tiles over 8 waves with 64-byte
// stages (two workgroups per CU), and large float32 ones 256x256 tiles over
// 8 waves, two per SIMD (half the operand bytes per flop of 128x128, and one
// wave's waits overlap the other's MFMAs).
template <typename Tin>
static hipError_t gemm_dt(const GemmDesc& g, hipStream_t st) {
    const int64_t mt128 = (g.M + 127) / 128;
    if constexpr (sizeof(Tin) == 2) {
        // bfloat16, measured on the DeiT-Base layer's products (50432 rows):
        // 64-byte stages, three in flight, and two workgroups per CU (72 KB
        // of LDS each) beat 128-byte stages two deep, which leave the loads'
        // latency exposed (fc1 + GELU 446 -> 407 us, the dense fc2 320 ->
        // 302); 256x128 over eight waves then beat every other tile of that
        // kind for the long products with N >= 512 (the pair y product, N =
        // 768, K = 384: 67 -> 58 us against 128x256) and for the long-K ones
        // with 128 < N <= 512 (the pair [t|u_a|u_b] product, N = 384, K =
        // 3072: 180 -> 173 us against 128x128 over four waves)
        const int64_t mnk = g.M * static_cast<int64_t>(g.N) * g.K;
        if (g.N >= 512 && (mnk >= (int64_t{1} << 35) || g.M >= 16384))
            return gemm_cfg<Tin, 256, 128, 4, 2, 3, 64>(g, st);
        if (g.N > 128 && g.N <= 512 && g.K >= 1024 && g.M >= 16384)
            return gemm_cfg<Tin, 256, 128, 4, 2, 3, 64>(g, st);
        if (g.N >= 1024 && g.K <= 512) return gemm_cfg<Tin, 128, 128, 4, 2, 2>(g, st);
        // long k rows (2 KB or more) over a few hundred 64x64 tiles (e.g. the
        // pair products of an adaptive layer at DeiT-Small widths, 28 -> 20
        // us): four stages in flight; with more tiles, 128x128 over 8 waves
        // (the DeiT-Small dense fc2, 35 -> 32 us)
        if (g.K >= 1024 && g.N > 128 && g.N <= 512) {
            const int64_t t64 = ((g.M + 63) / 64 + (g.seg_offsets != nullptr ? g.nseg : 0)) * ((g.N + 63) / 64);
            if (t64 <= 1024) return gemm_cfg<Tin, 64, 64, 2, 2, 4>(g, st);
            return gemm_cfg<Tin, 128, 128, 4, 2, 2>(g, st);
        }
    }
    if (g.N >= 1024 && ((g.M + 255) / 256) * ((g.N + 255) / 256) >= 1024)
        return gemm_cfg<Tin, 256, 256, 4, 2, 2>(g, st);
    if (g.N <= 32) return gemm_cfg<Tin, 128, 32, 4, 1, 3>(g, st);
    if (g.N <= 64) return gemm_cfg<Tin, 128, 64, 4, 1, 3>(g, st);
    // long k rows (2 KB or more: a float32 stage holds half the k of a bf16 one)
    const int64_t kbytes = static_cast<int64_t>(g.K) * static_cast<int64_t>(sizeof(Tin));
    if (g.N <= 128 && kbytes >= 2048) return gemm_cfg<Tin, 64, 64, 2, 2, 4>(g, st);
    if (mt128 * ((g.N + 127) / 128) < 2048) return gemm_cfg<Tin, 64, 128, 2, 2, 2>(g, st);
    return gemm_cfg<Tin, 128, 128, 2, 2, 2>(g, st);
}

hipError_t launch_gemm(int dtype, const GemmDesc& g, hipStream_t st) {
    if (dtype == 0) return gemm_dt<float>(g, st);
    return gemm_dt<bf16_bits>(g, st);
}

}  // namespace clearmoe
