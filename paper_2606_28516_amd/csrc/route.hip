// Router of the CLEAR-MoE layer: logits, top-k, renormalised gates and the
// per-tile expert histogram, fused in one pass over x.
//
// Linear router with bias (Sec. III Phase 4; the bias is what makes Table
// C5's parameter count), top-1 = Algorithm 3's argmax, top-k with the softmax
// of the selected logits renormalised.
//
// Precision: the logits are accumulated in double.  bf16*bf16 and f32*f32
// products are exact in double, so the only rounding is the double sum; the
// expert choice is therefore the exact one for every token whose top-k
// margin exceeds ~1e-13, which makes the choice reproducible against any
// double-precision evaluation of the same dot products.
//
// Layout / mapping (gfx950, wave64):
//   * one workgroup = 256 tokens = 256 threads, one token per thread;
//   * the token rows are staged through LDS in 128-byte column chunks (16-byte
//     coalesced global loads, 144-byte padded LDS rows: conflict-free 16-byte
//     reads of a row per lane), double buffered;
//   * the router weights are pre-widened to double and transposed
//     (wgT[d][e]), so for each column d the E weights are one wave-uniform
//     64-byte scalar load and each FMA takes its weight from SGPRs;
//   * the histogram is E ballots per wave, summed over the 4 waves in LDS.
#include "kernels.h"

namespace clearmoe {

template <typename Tin>
__global__ void k_router_weights_f64(const Tin* __restrict__ Wg, int D, int E, int emax, int Dpad,
                                     double* __restrict__ wgT) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= Dpad * emax) return;
    const int d = i / emax, e = i % emax;
    double v = 0.0;
    if (d < D && e < E) v = static_cast<double>(Elem<Tin>::load(Wg, static_cast<int64_t>(e) * D + d));
    wgT[i] = v;
}

template <typename Tin, int EMAX>
__global__ __launch_bounds__(kRouteTile, 2) void k_route(
    const Tin* __restrict__ x, const double* __restrict__ wgT, const float* __restrict__ bg,
    int64_t T, int D, int Dpad, int E, int k, int32_t* __restrict__ idx,
    float* __restrict__ gate, int32_t* __restrict__ tile_counts) {
    constexpr int STRIDE = kRouteChunkBytes + 16;
    constexpr int PER16 = Elem<Tin>::per16;
    constexpr int EPC = kRouteChunkBytes / static_cast<int>(sizeof(Tin));  // elements / chunk
    constexpr int PIECES = kRouteChunkBytes / 16;                          // 16B pieces / row
    constexpr int LOADS = PIECES;                                          // pieces / thread
    __shared__ __align__(16) unsigned char sx[2][kRouteTile * STRIDE];
    __shared__ int s_wcnt[kRouteTile / 64][EMAX];

    const int tid = threadIdx.x;
    const int64_t t0 = static_cast<int64_t>(blockIdx.x) * kRouteTile;
    const int64_t left = T - t0;
    const int rows = left < kRouteTile ? static_cast<int>(left) : kRouteTile;
    const int nchunk = Dpad / EPC;

    double acc[EMAX];
#pragma unroll
    for (int e = 0; e < EMAX; ++e) acc[e] = 0.0;

    uint4 reg[LOADS];
    auto gload = [&](int c) {
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            const int piece = tid + i * kRouteTile;
            const int row = piece / PIECES, pc = piece % PIECES;
            const int col = c * EPC + pc * PER16;
            uint4 v = make_uint4(0u, 0u, 0u, 0u);
            if (row < rows && col < D)
                v = *reinterpret_cast<const uint4*>(x + (t0 + row) * D + col);
            reg[i] = v;
        }
    };
    auto lstore = [&](int buf) {
#pragma unroll
        for (int i = 0; i < LOADS; ++i) {
            const int piece = tid + i * kRouteTile;
            const int row = piece / PIECES, pc = piece % PIECES;
            *reinterpret_cast<uint4*>(&sx[buf][row * STRIDE + pc * 16]) = reg[i];
        }
    };

    gload(0);
    lstore(0);
    __syncthreads();
    for (int c = 0; c < nchunk; ++c) {
        const int buf = c & 1;
        if (c + 1 < nchunk) gload(c + 1);
        const unsigned char* myrow = &sx[buf][tid * STRIDE];
#pragma unroll
        for (int pc = 0; pc < PIECES; ++pc) {
            const uint4 v = *reinterpret_cast<const uint4*>(myrow + pc * 16);
            Tin vals[PER16];
            __builtin_memcpy(vals, &v, 16);
#pragma unroll
            for (int u = 0; u < PER16; ++u) {
                const double xd = static_cast<double>(Elem<Tin>::to_f32(vals[u]));
                const double* w = wgT + static_cast<int64_t>(c * EPC + pc * PER16 + u) * EMAX;
#pragma unroll
                for (int e = 0; e < EMAX; ++e) acc[e] = __builtin_fma(xd, w[e], acc[e]);
            }
        }
        if (c + 1 < nchunk) lstore(buf ^ 1);
        __syncthreads();
    }

    const bool valid = tid < rows;
    const int64_t t = t0 + tid;
#pragma unroll
    for (int e = 0; e < EMAX; ++e)
        if (bg != nullptr && e < E) acc[e] += static_cast<double>(bg[e]);

    // Top-k: logit descending, ties to the lower expert index (strict '>'
    // while scanning upwards).  The first untaken expert always seeds the
    // scan, so a choice is made even for NaN logits.
    uint64_t taken = 0;
    double top = 0.0, den = 0.0;
    for (int j = 0; j < k; ++j) {
        int best = -1;
        double bv = 0.0;
#pragma unroll
        for (int e = 0; e < EMAX; ++e) {
            if (e < E && !((taken >> e) & 1ull) && (best < 0 || acc[e] > bv)) {
                best = e;
                bv = acc[e];
            }
        }
        taken |= 1ull << best;
        if (j == 0) top = bv;
        if (k > 1) den += exp(bv - top);
        if (valid) idx[t * k + j] = best;
    }
    if (valid) {
        if (k == 1) {
            gate[t] = 1.0f;
        } else {
            uint64_t tk = 0;
            for (int j = 0; j < k; ++j) {
                int best = -1;
                double bv = 0.0;
#pragma unroll
                for (int e = 0; e < EMAX; ++e) {
                    if (e < E && !((tk >> e) & 1ull) && (best < 0 || acc[e] > bv)) {
                        best = e;
                        bv = acc[e];
                    }
                }
                tk |= 1ull << best;
                gate[t * k + j] = static_cast<float>(exp(bv - top) / den);
            }
        }
    }

    if (tile_counts != nullptr) {
        const int lane = tid & 63, w = tid >> 6;
        for (int e = 0; e < E; ++e) {
            const uint64_t m = __ballot(valid && ((taken >> e) & 1ull));
            if (lane == 0) s_wcnt[w][e] = __popcll(m);
        }
        __syncthreads();
        if (tid < E) {
            int s = 0;
#pragma unroll
            for (int i = 0; i < kRouteTile / 64; ++i) s += s_wcnt[i][tid];
            tile_counts[static_cast<int64_t>(blockIdx.x) * E + tid] = s;
        }
    }
}

hipError_t launch_router_weights_f64(int dtype, const void* Wg, int D, int E, int emax, int Dpad,
                                     double* wgT, hipStream_t st) {
    const int n = Dpad * emax;
    const int blocks = (n + 255) / 256;
    if (dtype == 0)
        k_router_weights_f64<float><<<blocks, 256, 0, st>>>(static_cast<const float*>(Wg), D, E,
                                                             emax, Dpad, wgT);
    else
        k_router_weights_f64<bf16_bits><<<blocks, 256, 0, st>>>(
            static_cast<const bf16_bits*>(Wg), D, E, emax, Dpad, wgT);
    return hipGetLastError();
}

template <typename Tin>
static hipError_t route_dt(const Tin* x, const double* wgT, const float* bg, int64_t T, int D,
                           int Dpad, int E, int emax, int k, int32_t* idx, float* gate,
                           int32_t* tc, hipStream_t st) {
    const int64_t blocks = route_tiles(T);
    if (blocks == 0) return hipSuccess;
#define CLEARMOE_ROUTE_CASE(EM)                                                                  \
    case EM:                                                                                     \
        k_route<Tin, EM><<<dim3(static_cast<unsigned>(blocks)), kRouteTile, 0, st>>>(           \
            x, wgT, bg, T, D, Dpad, E, k, idx, gate, tc);                                        \
        break;
    switch (emax) {
        CLEARMOE_ROUTE_CASE(1)
        CLEARMOE_ROUTE_CASE(2)
        CLEARMOE_ROUTE_CASE(3)
        CLEARMOE_ROUTE_CASE(4)
        CLEARMOE_ROUTE_CASE(5)
        CLEARMOE_ROUTE_CASE(6)
        CLEARMOE_ROUTE_CASE(7)
        CLEARMOE_ROUTE_CASE(8)
        CLEARMOE_ROUTE_CASE(16)
        CLEARMOE_ROUTE_CASE(32)
        CLEARMOE_ROUTE_CASE(64)
        default:
            return hipErrorInvalidValue;
    }
#undef CLEARMOE_ROUTE_CASE
    return hipGetLastError();
}

hipError_t launch_route(int dtype, const void* x, const double* wgT, const float* bg, int64_t T,
                        int D, int Dpad, int E, int emax, int k, int32_t* idx, float* gate,
                        int32_t* tile_counts, hipStream_t st) {
    if (dtype == 0)
        return route_dt<float>(static_cast<const float*>(x), wgT, bg, T, D, Dpad, E, emax, k, idx,
                               gate, tile_counts, st);
    return route_dt<bf16_bits>(static_cast<const bf16_bits*>(x), wgT, bg, T, D, Dpad, E, emax, k,
                               idx, gate, tile_counts, st);
}

}  // namespace clearmoe
