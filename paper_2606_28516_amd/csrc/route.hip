// Router of the CLEAR-MoE layer: logits, top-k, renormalised gates and the
// per-tile expert histogram, fused in one pass over x.
//
// Linear router with bias (Sec. III Phase 4; the bias is what makes Table
// C5's parameter count), top-1 = Algorithm 3's argmax, top-k with the softmax
// of the selected logits renormalised; ties go to the lower expert index.
//
// Exact decisions at MFMA speed.  The logits are accumulated by MFMA in
// float32 (bf16 x bf16 products are exact in float32) in partial sums of
// kPart columns, which are added in double.  A second MFMA over |x| and |w|
// gives S_e = sum_d |x_d w_ed|; the float32 error of each partial is at most
// (kPart + 8) u S_partial, so every logit is within beta = 2 (kPart + 8) u S_e
// of its exact value (u = 2^-24; the factor 2 covers products that float32
// inputs round, and leaves slack for the MFMA's internal order).  A token
// whose consecutive top-(k+1) gaps all exceed 2 beta has provably the same
// top-k, in the same order, as the exact logits.  Every other token (near
// ties, a small fraction) is recomputed in double by its whole wave (64 lanes
// split D, butterfly sum), so the choice is the exact one for every token
// whose margin exceeds the double rounding of a D-term sum.  Gates use the
// same logits (double for the recomputed tokens, certified float32 sums of
// double partials for the others).
//
// Mapping (gfx950, wave64): a workgroup of 4 waves routes 256 tokens, a wave
// 64 tokens as four 16-token MFMA column blocks: v_mfma_f32_16x16x32_bf16
// (f32 input: v_mfma_f32_16x16x4f32 over four k-steps) with A = 16 router rows
// and B = 16 token rows, each lane loading 16 contiguous bytes of a token row.
// The 16 x 16 results go through LDS so that each lane owns one token for the
// top-k, gates and the ballot histogram.
#include <type_traits>

#include "kernels.h"

namespace clearmoe {

#ifndef KPRE
#define KPRE 4   // steps of x / router rows in flight per wave
#endif

__device__ __attribute__((aligned(16))) const uint32_t g_route_zero[4] = {0u, 0u, 0u, 0u};

template <typename Tin> struct RouteMfma;
template <> struct RouteMfma<bf16_bits> {
    static constexpr int kstep = 32;   // d per 16-byte-per-lane step (4 lane groups x 8)
    static constexpr int kpart = 64;   // columns per float32 partial sum of a logit
    __device__ static void step(const uint4& a, const uint4& b, f32x4& c) {
        c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                     __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }
    __device__ static uint4 absv(uint4 v) {
        return make_uint4(v.x & 0x7fff7fffu, v.y & 0x7fff7fffu, v.z & 0x7fff7fffu,
                          v.w & 0x7fff7fffu);
    }
};
template <> struct RouteMfma<float> {
    static constexpr int kstep = 16;   // 4 lane groups x 4 floats, four MFMAs of k = 4
    static constexpr int kpart = 32;
    __device__ static void step(const uint4& a, const uint4& b, f32x4& c) {
        const f32x4 av = __builtin_bit_cast(f32x4, a);
        const f32x4 bv = __builtin_bit_cast(f32x4, b);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(av[0], bv[0], c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(av[1], bv[1], c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(av[2], bv[2], c, 0, 0, 0);
        c = __builtin_amdgcn_mfma_f32_16x16x4f32(av[3], bv[3], c, 0, 0, 0);
    }
    __device__ static uint4 absv(uint4 v) {
        return make_uint4(v.x & 0x7fffffffu, v.y & 0x7fffffffu, v.z & 0x7fffffffu,
                          v.w & 0x7fffffffu);
    }
};

// Element s of a 16-byte piece, widened to double (register shifts only: s
// is a compile-time constant after unrolling).
template <typename Tin> __device__ double elem_f64(const uint4& v, int s);
template <>
__device__ __forceinline__ double elem_f64<bf16_bits>(const uint4& v, int s) {
    const uint32_t w = s < 2 ? v.x : s < 4 ? v.y : s < 6 ? v.z : v.w;
    return static_cast<double>(__uint_as_float((s & 1) ? (w & 0xffff0000u) : (w << 16)));
}
template <>
__device__ __forceinline__ double elem_f64<float>(const uint4& v, int s) {
    const uint32_t w = s == 0 ? v.x : s == 1 ? v.y : s == 2 ? v.z : v.w;
    return static_cast<double>(__uint_as_float(w));
}

// One selection step over lg[0..E): the best expert not in `taken`
// (logit descending, ties to the lower index: strict '>' while scanning up).
// The first untaken expert seeds the scan, so NaN logits still give a choice.
template <int EP>
__device__ __forceinline__ int pick(const double (&lg)[EP], int E, uint64_t taken, double& bv) {
    int best = -1;
    bv = 0.0;
#pragma unroll
    for (int e = 0; e < EP; ++e) {
        if (e < E && !((taken >> e) & 1ull) && (best < 0 || lg[e] > bv)) {
            best = e;
            bv = lg[e];
        }
    }
    return best;
}

// Smallest gap between consecutive logits of the sorted top-min(k+1, E): the
// margin that decides both the selected set and the slot order.
template <int EP>
__device__ __forceinline__ double topk_gap(const double (&lg)[EP], int E, int k) {
    uint64_t taken = 0;
    double prev = 0.0, gap = __builtin_inf();
    const int m = k < E ? k + 1 : E;
    for (int j = 0; j < m; ++j) {
        double bv;
        const int best = pick<EP>(lg, E, taken, bv);
        taken |= 1ull << best;
        if (j > 0) gap = fmin(gap, prev - bv);
        prev = bv;
    }
    return gap;
}

// Double exp as one out-of-line routine: the choice code below calls it from
// unrolled loops, and a single copy keeps the kernels' code (and so their
// cold instruction-cache misses) small.
__device__ __attribute__((noinline)) double exp_ool(double v) { return exp(v); }

// Largest softmax probability of a token over its E logits,
// 1 / sum_e exp(l_e - l_max): the confidence of the adaptive router.
template <int EP>
__device__ __forceinline__ double route_confidence(const double (&lg)[EP], int E) {
    double lmax = lg[0];
#pragma unroll
    for (int e = 1; e < EP; ++e)
        if (e < E && lg[e] > lmax) lmax = lg[e];
    double den = 0.0;
#pragma unroll
    for (int e = 0; e < EP; ++e)
        if (e < E) den += exp_ool(lg[e] - lmax);
    return 1.0 / den;
}

// Choice of one token from its logits (descending, ties to the lower index):
// the top k, or, adaptive (k = 2 slots), top-1 when the confidence reaches
// tau and top-2 otherwise, the unused second slot being expert -1 with gate
// 0.  Gates: renorm != 0, the softmax of the selected logits renormalised
// over them (k = 1: gate 1); renorm == 0, the selected experts' probabilities
// under the softmax over all E logits (their sum is below 1 unless every
// expert is selected).  Writes idx/gate of token t; returns the bit set of
// the chosen experts.
template <int EP>
__device__ __forceinline__ uint64_t route_select(const double (&lg)[EP], int E, int k,
                                                 int adaptive, int renorm, double tau, int64_t t,
                                                 int32_t* __restrict__ idx,
                                                 float* __restrict__ gate) {
    // the largest probability under the softmax over all E (adaptive choice;
    // renorm == 0: an expert's gate is exp(l - l_max) times it)
    const double conf = (adaptive || !renorm) ? route_confidence<EP>(lg, E) : 1.0;
    const int kk = (adaptive && conf >= tau) ? 1 : k;
    if (kk == 2) {
        // two experts: gates 1 / (1 + e1) and e1 / (1 + e1), e1 = exp(l1 - l0)
        // (the general loop's arithmetic: exp(0) = 1 exactly), one exp
        double v0, v1;
        const int b0 = pick<EP>(lg, E, 0ull, v0);
        const int b1 = pick<EP>(lg, E, 1ull << b0, v1);
        const double e1 = exp_ool(v1 - v0);
        const double den = renorm ? 1.0 + e1 : 1.0 / conf;
        idx[t * k] = b0;
        idx[t * k + 1] = b1;
        gate[t * k] = static_cast<float>(1.0 / den);
        gate[t * k + 1] = static_cast<float>(e1 / den);   // kk == 2 only when k == 2
        return (1ull << b0) | (1ull << b1);
    }
    uint64_t mine = 0;
    double top = 0.0, den = 0.0;
    for (int j = 0; j < kk; ++j) {
        double bv;
        const int best = pick<EP>(lg, E, mine, bv);
        mine |= 1ull << best;
        if (j == 0) top = bv;
        if (kk > 1 && renorm) den += exp_ool(bv - top);   // one expert: its gate is 1
        idx[t * k + j] = best;
    }
    if (!renorm) den = 1.0 / conf;           // top is the largest logit
    if (kk == 1) {
        gate[t * k] = renorm ? 1.0f : static_cast<float>(conf);
    } else {
        uint64_t tk = 0;
        for (int j = 0; j < kk; ++j) {
            double bv;
            const int best = pick<EP>(lg, E, tk, bv);
            tk |= 1ull << best;
            gate[t * k + j] = static_cast<float>(exp_ool(bv - top) / den);
        }
    }
    for (int j = kk; j < k; ++j) {          // adaptive top-1: empty second slot
        idx[t * k + j] = -1;
        gate[t * k + j] = 0.0f;
    }
    return mine;
}

// 16 bytes per lane, global -> LDS at m0 + 16 * lane.  Inline asm, issued
// before any other load of the wave: every later wait of the wave (the
// compiler's, in issue order) also covers it.
__device__ __forceinline__ void route_dma16(const void* gptr, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                 :
                 : "s"(lds_addr), "v"(gptr)
                 : "memory", "m0");
}

typedef __attribute__((address_space(3))) uint32_t route_lds_word;

// w_lds > 0: the router matrix (E x D, w_lds bytes of dynamic LDS) is copied to
// LDS for the exact recompute of uncertified tokens.
template <typename Tin, int EG, int NB, int KP>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(EG == 1 ? 2 : 1)))
void k_route(
    const Tin* __restrict__ x, const Tin* __restrict__ Wg, const float* __restrict__ bg, int64_t T,
    int D, int E, int k, int adaptive, int renorm, double tau, int dense_stride, int32_t* __restrict__ idx,
    float* __restrict__ gate, int32_t* __restrict__ tile_counts, int w_lds) {
    extern __shared__ __attribute__((aligned(16))) unsigned char s_w[];
    constexpr int EP = 16 * EG;                      // experts padded to MFMA rows
    constexpr int PER16 = Elem<Tin>::per16;
    constexpr int KS = RouteMfma<Tin>::kstep;
    constexpr int kPart = RouteMfma<Tin>::kpart;
    constexpr int kWaves = 4;
    constexpr int kTok = 16 * NB;                    // tokens per wave
    constexpr int kTile = kWaves * kTok;             // tokens per workgroup = histogram tile
    static_assert(kTile == kRouteTile || kTile == kSmallTile, "histogram tile sizes");
    __shared__ double s_l[kWaves][64][17];           // kTok rows; 64 for the recompute's sums
    __shared__ float s_s[kWaves][kTok][4 * EG + 1];
    __shared__ int s_wcnt[kWaves][64];
    __shared__ double s_fb[kWaves][4][EP];           // recomputed logits of a batch

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int col = lane & 15, grp = lane >> 4;
    const int64_t tw = static_cast<int64_t>(blockIdx.x) * kTile + w * kTok;  // wave's first token
    // this tile's x rows and the router rows as raw buffers (zeros outside)
    constexpr int esz = static_cast<int>(sizeof(Tin));
    const int64_t tile0 = static_cast<int64_t>(blockIdx.x) * kTile;
    const int rows = static_cast<int>(T - tile0 < kTile ? T - tile0 : kTile);
    const __amdgpu_buffer_rsrc_t rx = raw_rsrc(x + tile0 * D, static_cast<int64_t>(rows) * D * esz);
    const __amdgpu_buffer_rsrc_t rw = raw_rsrc(Wg, static_cast<int64_t>(E) * D * esz);
    __shared__ double bgv[EP];                       // router bias, loaded up front (read
    if (tid < EP)                                    // after the barrier past the transposes)
        bgv[tid] = (bg != nullptr && tid < E) ? static_cast<double>(bg[tid]) : 0.0;

    if (w_lds > 0) {                               // router rows -> LDS (read after a barrier)
        const int64_t wbytes = static_cast<int64_t>(E) * D * static_cast<int>(sizeof(Tin));
        const uint32_t base_l =
            static_cast<uint32_t>(reinterpret_cast<uintptr_t>((route_lds_word*)s_w));
        for (int base = w * 64; base * 16 < w_lds; base += 64 * kWaves) {
            const int64_t off = static_cast<int64_t>(base + lane) * 16;
            const void* src = off < wbytes ? static_cast<const void*>(
                                                 reinterpret_cast<const unsigned char*>(Wg) + off)
                                           : static_cast<const void*>(g_route_zero);
            route_dma16(src, __builtin_amdgcn_readfirstlane(base_l + base * 16));
        }
    }

    f32x4 acc[EG][NB], aab[EG][NB];
    double lacc[EG][NB][4];            // double sums of the float32 partials
#pragma unroll
    for (int g = 0; g < EG; ++g)
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                acc[g][b][v] = aab[g][b][v] = 0.0f;
                lacc[g][b][v] = 0.0;
            }

    // Loads of MFMA k-steps (KS columns of d each) for the wave's NB token
    // blocks and the router rows, two k-steps per ring step: the two 16-byte
    // loads a lane makes from one row cover the two 64-byte halves of a
    // 128-byte line and are issued back to back.  A ring of kPre / 2 ring
    // steps keeps several in flight; the loop is branch-free (columns past D
    // and rows past the tile read zeros from the raw buffers), so the
    // compiler's waits stay per round instead of per step.  Every kPart
    // columns the float32 partials move into double.
    constexpr int kPre = KP;
    static_assert(kPre % 2 == 0 && (kPre * KS) % kPart == 0 && (2 * KS) % kPart == 0,
                  "partials align with ring steps");
    const int nsteps = (D + KS - 1) / KS;
    constexpr int kP = kPre / 2;
    uint4 xr[kP][NB][2], wr[kP][EG][2];
    auto load_step = [&](int s, uint4 (&xv)[NB][2], uint4 (&wv)[EG][2]) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int dd = (2 * s + h) * KS + grp * PER16;
            const bool din = dd < D;
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const int tr = w * kTok + 16 * b + col;
                xv[b][h] = raw_load16(rx, (din && tr < rows) ? static_cast<uint32_t>((tr * D + dd) * esz) : kRawOob);
            }
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int dd = (2 * s + h) * KS + grp * PER16;
            const bool din = dd < D;
#pragma unroll
            for (int g = 0; g < EG; ++g) {
                const int e = 16 * g + col;
                wv[g][h] = raw_load16(rw, (din && e < E) ? static_cast<uint32_t>((e * D + dd) * esz) : kRawOob);
            }
        }
    };
    const int nround2 = (nsteps + 2 * kP - 1) / (2 * kP);
#pragma unroll
    for (int i = 0; i < kP; ++i) load_step(i, xr[i], wr[i]);
    for (int o = 0; o < nround2; ++o) {
#pragma unroll
        for (int i = 0; i < kP; ++i) {
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int g = 0; g < EG; ++g) {
                const uint4 wa = RouteMfma<Tin>::absv(wr[i][g][h]);
#pragma unroll
                for (int b = 0; b < NB; ++b) {
                    RouteMfma<Tin>::step(wr[i][g][h], xr[i][b][h], acc[g][b]);
                    RouteMfma<Tin>::step(wa, RouteMfma<Tin>::absv(xr[i][b][h]), aab[g][b]);
                }
            }
            load_step((o + 1) * kP + i, xr[i], wr[i]);
            if (((i + 1) * 2 * KS) % kPart == 0) {
#pragma unroll
                for (int g = 0; g < EG; ++g)
#pragma unroll
                    for (int b = 0; b < NB; ++b)
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            lacc[g][b][v] += static_cast<double>(acc[g][b][v]);
                            acc[g][b][v] = 0.0f;
                        }
            }
        }
    }
    // C of a 16x16 MFMA: lane holds column lane%16 (token), rows 4*(lane/16)+v
    // (experts).  Through LDS, one 16-expert group at a time, each of the
    // wave's first kTok lanes takes the logits of one token; for S only each
    // lane's maximum over its four experts is exchanged.
    const int64_t t = tw + lane;
    // a class token (dense path) takes no expert: no choice to certify
    const bool cls = dense_stride > 0 && t % dense_stride == 0;
    const bool valid = lane < kTok && t < T && !cls;
    const int tl = lane < kTok ? lane : kTok - 1;    // lanes past the wave's tokens idle
    double lg[EP];
#pragma unroll
    for (int g = 0; g < EG; ++g) {
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
            for (int v = 0; v < 4; ++v) s_l[w][16 * b + col][4 * grp + v] = lacc[g][b][v];
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            float m = 0.0f;
#pragma unroll
            for (int v = 0; v < 4; ++v)
                if (16 * g + 4 * grp + v < E) m = fmaxf(m, aab[g][b][v]);
            s_s[w][16 * b + col][4 * g + grp] = m;
        }
        // s_l[w] and s_s[w] are this wave's own rows: a wave-level barrier
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int e = 0; e < 16; ++e) lg[16 * g + e] = s_l[w][tl][e];
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    // the bias (written by the first threads) and the router rows in LDS
    // (every wave's copy has landed: its later loads have) are read below
    __syncthreads();
    float smax = 0.0f;
#pragma unroll
    for (int i = 0; i < 4 * EG; ++i) smax = fmaxf(smax, s_s[w][tl][i]);
#pragma unroll
    for (int e = 0; e < EP; ++e) lg[e] += bgv[e];
    // Rounding bound of every logit (S itself rounded up by 1%).
    const double beta = 2.0 * (kPart + 8) * 0x1p-24 * static_cast<double>(smax) * 1.01;
    bool certain = topk_gap<EP>(lg, E, k) > 2.0 * beta;
    if (adaptive && certain && tau > 0.0) {
        // log of the confidence moves by at most 2 beta (l_max and the
        // log-sum-exp by beta each): decide only outside that band
        const double lp = log(route_confidence<EP>(lg, E));
        certain = fabs(lp - log(tau)) > 2.0 * beta + 1e-12;
    }

    // ---- exact recompute in double of the tokens that are not certified.
    //      A batch takes nb = 1, 2 or 4 of them (as many as are left, up to
    //      4); lane group q = lane / G (G = 64 / nb lanes) takes the q-th, lane
    //      r = lane % G its 16-byte chunks r, r + G, ... (the loads of a pass
    //      issued first, each x chunk widened once), router rows from LDS when
    //      they fit; a G-lane butterfly sums each group, and the sums reach the
    //      owner lane through LDS.  One uncertified token (the usual case)
    //      thus has the whole wave.  The loops over experts and chunks are
    //      left rolled: this path is rare and runs from a cold instruction
    //      cache, so its code is kept small.
    uint64_t todo = __ballot(valid && !certain);
    while (todo != 0ull) {
        const int left = __popcll(todo);
        const int nb = left >= 4 ? 4 : (left >= 2 ? 2 : 1);
        const int G = 64 / nb;
        int myq = -1, src_tok[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            src_tok[q] = -1;
            if (q < nb) {
                const int o = __ffsll(static_cast<long long>(todo)) - 1;
                todo &= todo - 1ull;
                src_tok[q] = o;
                if (lane == o) myq = q;
            }
        }
        const int q = lane / G, r = lane - q * G;
        const int mine_tok = q == 0 ? src_tok[0] : q == 1 ? src_tok[1] : q == 2 ? src_tok[2] : src_tok[3];
        const int trow = w * kTok + mine_tok;          // row within the tile
        const int nch = D / PER16;                     // 16-byte chunks of a row
        // all experts in one pass over the lane's chunks (x loaded and widened
        // once per chunk), then one butterfly for all of them, so the
        // experts' shuffles overlap instead of forming E dependent chains
        double part[EP];
#pragma unroll
        for (int e = 0; e < EP; ++e) part[e] = 0.0;
#pragma unroll 1
        for (int c = r; c - r < nch; c += G) {
            const bool in = mine_tok >= 0 && c < nch;
            const uint4 xv = raw_load16(rx, in ? static_cast<uint32_t>((trow * D + c * PER16) * esz) : kRawOob);
            const int cc = c < nch ? c : 0;            // past the row: zero x, any valid W chunk
            double xd[PER16];
#pragma unroll
            for (int i = 0; i < PER16; ++i) xd[i] = elem_f64<Tin>(xv, i);
#pragma unroll
            for (int e = 0; e < EP; ++e) {
                if (e < E) {                           // uniform
                    const int64_t at = static_cast<int64_t>(e) * D + cc * PER16;
                    uint4 wv;
                    if (w_lds > 0)
                        wv = *reinterpret_cast<const uint4*>(s_w + at * static_cast<int64_t>(sizeof(Tin)));
                    else
                        wv = raw_load16(rw, static_cast<uint32_t>(at * esz));
#pragma unroll
                    for (int i = 0; i < PER16; ++i)
                        part[e] = __builtin_fma(xd[i], elem_f64<Tin>(wv, i), part[e]);
                }
            }
        }
        // sums over each group's G lanes through LDS (this wave's transpose
        // rows, free by now): lane (q, e) adds its group's column e
        double* red = &s_l[w][0][0];                  // [64 lanes][16 experts], pitch 17
#pragma unroll
        for (int g = 0; g < EG; ++g) {
#pragma unroll
            for (int e = 0; e < 16; ++e)
                if (16 * g + e < E) red[lane * 17 + e] = part[16 * g + e];
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            if (lane < 16 * nb) {
                const int qq = lane >> 4, e = lane & 15;
                if (16 * g + e < E) {
                    double acc = 0.0;
                    for (int j = 0; j < G; ++j) acc += red[(qq * G + j) * 17 + e];
                    s_fb[w][qq][16 * g + e] = acc;
                }
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        if (myq >= 0) {
#pragma unroll
            for (int e = 0; e < EP; ++e)
                if (e < E) lg[e] = s_fb[w][myq][e] + bgv[e];
        }
        __builtin_amdgcn_wave_barrier();
    }
    // ---- top-k (or adaptive top-1 / top-2), gates, outputs
    uint64_t mine = 0;
    if (valid) mine = route_select<EP>(lg, E, k, adaptive, renorm, tau, t, idx, gate);
    if (cls && lane < kTok && t < T) {
        for (int j = 0; j < k; ++j) {
            idx[t * k + j] = -1;
            gate[t * k + j] = 0.0f;
        }
    }
    if (tile_counts != nullptr) {
        for (int e = 0; e < E; ++e) {
            const uint64_t m = __ballot((mine >> e) & 1ull);
            if (lane == 0) s_wcnt[w][e] = __popcll(m);
        }
        __syncthreads();
        if (tid < E) {
            int s = 0;
#pragma unroll
            for (int i = 0; i < kWaves; ++i) s += s_wcnt[i][tid];
            tile_counts[static_cast<int64_t>(blockIdx.x) * E + tid] = s;
        }
    }
}

// ---------------------------------------------------------------------------
// MLP router (Sec. III Phase 4: one hidden layer, width d/6 in the paper):
//     hr = round_storage(GELU(x Wh^T + bh)),   l = hr Wo^T + bo,
// then the same top-k / adaptive choice as the linear router.  The hidden
// layer is rounded to the storage type (where a real deployment keeps it),
// and that rounding decides the logits to far more than the 1e-6 routing
// margin, so it must be taken on the exact pre-activation: both products run
// in double on the f64 MFMA (v_mfma_f64_16x16x4f64, the same 78.6 TFLOP/s as
// the vector unit, fed by 16-byte loads), GELU uses the double erf, and the
// rounding to bfloat16 is done straight from double (one rounding, ties to
// even).  Storage products are exact in double; only the summation order
// differs from a plain loop.
//
// Mapping: a workgroup of 4 waves routes 16 tokens; wave w forms hidden
// units [16 i, 16 i + 16) for i = w, w + 4, ... (one 16 x 16 f64 MFMA tile
// each), so a small token count still spreads over many waves.  In a D-chunk
// of 4 x per16 columns, lane l loads 16 bytes of token row l % 16 and of
// hidden row 16 i + l % 16 at column chunk l / 16, and feeds element s of
// them as MFMA k-index l / 16 in sub-step s: A = tokens x k, B = k x hidden
// units, the same (column, k) pairing on both sides.  Four chunks are loaded
// before their MFMAs, so a wave waits once per 4 chunks.  The f64 MFMA's
// result holds D[l / 16 + 4 v][l % 16] in value v of lane l.  The hidden
// values meet in LDS; wave g < EG then forms logits of experts [16 g, 16 g +
// 16), and the first 16 lanes of wave 0 take one token each for the choice.
typedef double f64x4 __attribute__((ext_vector_type(4)));
constexpr int kMlpTokens = 16;             // tokens per workgroup
constexpr int kMlpChunks = 4;              // 16-byte chunks in flight per lane
static_assert(kMlpHiddenMax == 256, "LDS plan of k_route_mlp");

__device__ __attribute__((noinline)) double mlp_gelu(double v) {
    return 0.5 * v * (1.0 + erf(v * 0.70710678118654752440));
}

// double -> nearest bfloat16 (ties to even), returned as the exact float.
__device__ __forceinline__ float round_to_bf16(double v) {
    uint64_t u = static_cast<uint64_t>(__double_as_longlong(v));
    u += ((uint64_t{1} << 44) - 1) + ((u >> 45) & 1);   // 45 of 52 mantissa bits dropped
    u &= ~((uint64_t{1} << 45) - 1);
    return static_cast<float>(__longlong_as_double(static_cast<long long>(u)));
}
template <typename Tin> __device__ float round_storage(double v);
template <> __device__ __forceinline__ float round_storage<bf16_bits>(double v) { return round_to_bf16(v); }
template <> __device__ __forceinline__ float round_storage<float>(double v) { return static_cast<float>(v); }

template <typename Tin, int EG>
__global__ __launch_bounds__(256) void k_route_mlp(
    const Tin* __restrict__ x, const Tin* __restrict__ Wh, const float* __restrict__ bh,
    const Tin* __restrict__ Wo, const float* __restrict__ bo, int64_t T, int D, int Hr, int E,
    int k, int adaptive, int renorm, double tau, int dense_stride, int32_t* __restrict__ idx,
    float* __restrict__ gate) {
    constexpr int EP = 16 * EG;
    static_assert(EG <= 4, "one wave per 16 experts");
    constexpr int PER16 = Elem<Tin>::per16;
    constexpr int KC = 4 * PER16;                   // columns per 16-byte-per-lane chunk
    __shared__ float s_hr[kMlpTokens][kMlpHiddenMax + 1];   // odd pitch: column reads spread
    __shared__ double s_lg[kMlpTokens][EP + 1];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int row = lane & 15, grp = lane >> 4;
    const int64_t t0 = static_cast<int64_t>(blockIdx.x) * kMlpTokens;
    constexpr int esz = static_cast<int>(sizeof(Tin));
    const int rows = static_cast<int>(T - t0 < kMlpTokens ? T - t0 : kMlpTokens);
    const __amdgpu_buffer_rsrc_t rx = raw_rsrc(x + t0 * D, static_cast<int64_t>(rows) * D * esz);
    const __amdgpu_buffer_rsrc_t rh = raw_rsrc(Wh, static_cast<int64_t>(Hr) * D * esz);

    // ---- hidden layer: one 16-unit tile per wave per pass
    for (int u0 = 16 * w; u0 < Hr; u0 += 64) {
        // two accumulators (even / odd sub-steps) halve the dependent chain
        f64x4 acc0 = f64x4{0.0, 0.0, 0.0, 0.0}, acc1 = acc0;
        const int u = u0 + row;
        for (int c0 = 0; c0 < D; c0 += kMlpChunks * KC) {
            uint4 xv[kMlpChunks], wv[kMlpChunks];
#pragma unroll
            for (int c = 0; c < kMlpChunks; ++c) {
                // D % PER16 == 0: a chunk is all in or out; rows past T or Hr
                // and columns past D read zeros from the raw buffers
                const int col = c0 + c * KC + grp * PER16;
                const bool cin = col < D;
                xv[c] = raw_load16(rx, (cin && row < rows) ? static_cast<uint32_t>((row * D + col) * esz) : kRawOob);
                wv[c] = raw_load16(rh, (cin && u < Hr) ? static_cast<uint32_t>((u * D + col) * esz) : kRawOob);
            }
#pragma unroll
            for (int c = 0; c < kMlpChunks; ++c)
#pragma unroll
                for (int s = 0; s < PER16; s += 2) {
                    acc0 = __builtin_amdgcn_mfma_f64_16x16x4f64(elem_f64<Tin>(xv[c], s),
                                                                elem_f64<Tin>(wv[c], s), acc0, 0, 0, 0);
                    acc1 = __builtin_amdgcn_mfma_f64_16x16x4f64(elem_f64<Tin>(xv[c], s + 1),
                                                                elem_f64<Tin>(wv[c], s + 1), acc1, 0, 0, 0);
                }
        }
        const f64x4 acc = acc0 + acc1;
        // + bias, GELU, one rounding to storage, into LDS (token-major)
        if (u < Hr) {
            const double b = bh != nullptr ? static_cast<double>(bh[u]) : 0.0;
#pragma unroll
            for (int v = 0; v < 4; ++v)              // result row = token grp + 4 v
                s_hr[grp + 4 * v][u] = round_storage<Tin>(mlp_gelu(acc[v] + b));
        }
    }
    __syncthreads();
    // ---- output layer l = hr Wo^T (+ bo below): wave g, experts [16 g, 16 g + 16)
    if (w < EG) {
        f64x4 acc = f64x4{0.0, 0.0, 0.0, 0.0};
        const int e = 16 * w + row;
        const Tin* orow = e < E ? Wo + static_cast<int64_t>(e) * Hr : nullptr;
        for (int j0 = 0; j0 < Hr; j0 += 4) {
            const int j = j0 + grp;
            const double a = j < Hr ? static_cast<double>(s_hr[row][j]) : 0.0;
            const double b = (orow != nullptr && j < Hr) ? static_cast<double>(Elem<Tin>::load(orow, j)) : 0.0;
            acc = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc, 0, 0, 0);
        }
#pragma unroll
        for (int v = 0; v < 4; ++v) s_lg[grp + 4 * v][16 * w + row] = acc[v];
    }
    __syncthreads();
    // ---- one token per lane (16 lanes of wave 0): choice, gates, outputs
    const int64_t t = t0 + lane;
    if (w == 0 && lane < kMlpTokens && t < T) {
        if (dense_stride > 0 && t % dense_stride == 0) {       // class token: no expert
            for (int j = 0; j < k; ++j) {
                idx[t * k + j] = -1;
                gate[t * k + j] = 0.0f;
            }
        } else {
            double lg[EP];
#pragma unroll
            for (int e = 0; e < EP; ++e)
                lg[e] = s_lg[lane][e] + ((bo != nullptr && e < E) ? static_cast<double>(bo[e]) : 0.0);
            (void)route_select<EP>(lg, E, k, adaptive, renorm, tau, t, idx, gate);
        }
    }
}

template <typename Tin>
static hipError_t route_mlp_dt(const Tin* x, const Tin* Wh, const float* bh, const Tin* Wo,
                               const float* bo, int64_t T, int D, int Hr, int E, int k,
                               int adaptive, int renorm, double tau, int dense_stride, int32_t* idx,
                               float* gate, hipStream_t st) {
    const int64_t blocks = (T + kMlpTokens - 1) / kMlpTokens;
    if (blocks == 0) return hipSuccess;
    const dim3 grid(static_cast<unsigned>(blocks));
    if (E <= 16)
        launch_kernel(k_route_mlp<Tin, 1>, grid, 256, 0, st, x, Wh, bh, Wo, bo, T, D, Hr, E, k, adaptive, renorm, tau,
                                                    dense_stride, idx, gate);
    else if (E <= 32)
        launch_kernel(k_route_mlp<Tin, 2>, grid, 256, 0, st, x, Wh, bh, Wo, bo, T, D, Hr, E, k, adaptive, renorm, tau,
                                                    dense_stride, idx, gate);
    else
        launch_kernel(k_route_mlp<Tin, 4>, grid, 256, 0, st, x, Wh, bh, Wo, bo, T, D, Hr, E, k, adaptive, renorm, tau,
                                                    dense_stride, idx, gate);
    return hipGetLastError();
}

hipError_t launch_route_mlp(int dtype, const void* x, const void* Wh, const float* bh,
                            const void* Wo, const float* bo, int64_t T, int D, int Hr, int E,
                            int k, int adaptive, int renorm, double tau, int dense_stride, int32_t* idx,
                            float* gate, hipStream_t st) {
    if (Hr < 1 || Hr > kMlpHiddenMax) return hipErrorInvalidValue;
    if (dtype == 0)
        return route_mlp_dt<float>(static_cast<const float*>(x), static_cast<const float*>(Wh), bh,
                                   static_cast<const float*>(Wo), bo, T, D, Hr, E, k, adaptive,
                                   renorm, tau, dense_stride, idx, gate, st);
    return route_mlp_dt<bf16_bits>(static_cast<const bf16_bits*>(x),
                                   static_cast<const bf16_bits*>(Wh), bh,
                                   static_cast<const bf16_bits*>(Wo), bo, T, D, Hr, E, k, adaptive,
                                   renorm, tau, dense_stride, idx, gate, st);
}

constexpr int64_t kRouteWLds = 32 * 1024;


template <typename Tin>
static hipError_t route_dt(const Tin* x, const Tin* Wg, const float* bg, int64_t T, int D, int E,
                           int k, int adaptive, int renorm, double tau, int dense_stride, int32_t* idx,
                           float* gate, int32_t* tc, hipStream_t st) {
    const int64_t blocks = hist_tiles(T, E);
    if (blocks == 0) return hipSuccess;
    const dim3 grid(static_cast<unsigned>(blocks));
    const bool small = hist_tile(T, E) == kSmallTile;   // implies E <= 16
    // the router rows go to LDS when they fit in kRouteWLds (whole 1 KB rounds)
    const int64_t wbytes = static_cast<int64_t>(E) * D * static_cast<int64_t>(sizeof(Tin));
    const int w_lds = wbytes <= kRouteWLds ? static_cast<int>((wbytes + 1023) / 1024 * 1024) : 0;
    if (small)
        launch_kernel(k_route<Tin, 1, 1, 12>, grid, 256, w_lds, st, x, Wg, bg, T, D, E, k, adaptive, renorm, tau,
                                                          dense_stride, idx, gate, tc, w_lds);
    else if (E <= 16)
        launch_kernel(k_route<Tin, 1, 4, KPRE>, grid, kRouteTile, w_lds, st, x, Wg, bg, T, D, E, k, adaptive,
                                                                   renorm, tau, dense_stride, idx, gate, tc,
                                                                   w_lds);
    else if (E <= 32)
        launch_kernel(k_route<Tin, 2, 4, KPRE>, grid, kRouteTile, w_lds, st, x, Wg, bg, T, D, E, k, adaptive,
                                                                   renorm, tau, dense_stride, idx, gate, tc,
                                                                   w_lds);
    else
        launch_kernel(k_route<Tin, 4, 4, KPRE>, grid, kRouteTile, w_lds, st, x, Wg, bg, T, D, E, k, adaptive,
                                                                   renorm, tau, dense_stride, idx, gate, tc,
                                                                   w_lds);
    return hipGetLastError();
}

hipError_t launch_route(int dtype, const void* x, const void* Wg, const float* bg, int64_t T,
                        int D, int E, int k, int adaptive, int renorm, double tau, int dense_stride,
                        int32_t* idx, float* gate, int32_t* tile_counts, hipStream_t st) {
    if (dtype == 0)
        return route_dt<float>(static_cast<const float*>(x), static_cast<const float*>(Wg), bg, T,
                               D, E, k, adaptive, renorm, tau, dense_stride, idx, gate, tile_counts, st);
    return route_dt<bf16_bits>(static_cast<const bf16_bits*>(x), static_cast<const bf16_bits*>(Wg),
                               bg, T, D, E, k, adaptive, renorm, tau, dense_stride, idx, gate, tile_counts,
                               st);
}

}  // namespace clearmoe
