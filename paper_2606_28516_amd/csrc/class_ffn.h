// Dense FFN of the class tokens (gfx950, bfloat16):
//     y[c] = GELU(x[c] W1^T + b1) W2^T + b2
// for the class rows c (every stride-th token, from token 0), which skip the
// router and take the original dense FFN (Sec. III; Table C6).  A block of 32
// class rows is split over P workgroups of 4 waves, part p taking a
// contiguous run of the hidden width's 128-unit chunks:
//   * phase 1: wave w forms z for its 32 units of the chunk (one 32x32 MFMA
//     tile over the D inputs, the class rows' x held in registers for the
//     whole pass), adds b1, applies GELU and rounds to bfloat16 into LDS;
//   * phase 2: wave w adds the chunk's 128 units to its 96 output columns of
//     y (three 32x32 tiles, float32 in registers), reading W2 directly;
//   * the next chunk's W1 rows are loaded during the GELU and phase 2, its
//     W2 rows during the next phase 1.
// With P = 1 the part writes y.  Otherwise every part stores its float32
// partial sums, and the last of the block's parts to arrive adds the P
// partials in part order (the same bits whichever part is last) and writes
// y.  Arrival is counted in one 64-bit word per block holding this launch's
// number and a count: the first arrival of a launch finds another number
// there (from an earlier launch, or memory never written) and restarts the
// count, so the words need no clearing between launches.  The parts' stores
// are released at agent scope before their arrival and acquired by the last
// part, wherever the parts run.
//
// A part is slow on its own (one CU streams its share of W1 and W2 with 32
// rows per load), so the pass is meant to run beside other work: inside the
// fused top-1 kernel's launch, on workgroups past its tiles, the class rows
// need no launch of their own and overlap the routed tokens' tiles.
#pragma once

#include "kernels.h"

namespace clearmoe {

struct ClassArgs {
    const bf16_bits* x;    // [T][D]
    const bf16_bits* W1;   // [H][D]
    const float* b1;       // [H] or null
    const bf16_bits* W2;   // [D][H]
    const float* b2;       // [D] or null
    bf16_bits* y;          // [T][D]: the class rows are written, nothing else
    int64_t ncls;          // class rows: ceil(T / stride)
    int64_t stride;        // tokens from one class row to the next
    int D, H;              // D <= 384 and H multiples of 8
    int nparts;            // P: workgroups per 32-row block
    int per;               // chunks per part (the last part may take fewer, never none)
    float* part;           // P > 1: [blocks][P][32 x 384] float32 partial sums
    uint64_t* count;       // P > 1: [blocks] arrival words (launch << 16 | arrivals)
    uint64_t launch;       // this launch's number: 1 .. 2^48 - 1
};

constexpr int kClsRows = 32;    // class rows per workgroup
constexpr int kClsChunk = 128;  // hidden units per chunk (32 per wave)
constexpr int kClsMaxD = 384;   // four waves x three 32-column tiles
constexpr int kClsKSteps = kClsMaxD / 16;
constexpr int kClsPartFloats = kClsRows * kClsMaxD;   // one part's partial sums
// Workspace of the split: partial sums and arrival words
constexpr size_t kClsPartBytes = static_cast<size_t>(2) << 20;
constexpr int kClsCountWords = 64;
constexpr int kClsMaxParts = 8;

constexpr int kClsZPitch = kClsChunk + 8;   // bf16 elements: conflict-free 16-byte reads
__host__ __device__ inline int class_hpad(int H) { return (H + kClsChunk - 1) / kClsChunk * kClsChunk; }
// LDS: [z chunk (bf16) | b1 (float32, zeros past H)]
__host__ __device__ inline size_t class_lds_bytes(int H) {
    return static_cast<size_t>(kClsRows) * kClsZPitch * 2 + static_cast<size_t>(class_hpad(H)) * 4;
}
inline int64_t class_blocks(int64_t ncls) { return (ncls + kClsRows - 1) / kClsRows; }

// LDS writes of this workgroup are visible to all its waves after the
// barrier; outstanding global loads stay in flight across it.
__device__ __forceinline__ void class_lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Workgroup j of the pass: block j / P, part j % P; lds holds
// class_lds_bytes(c.H) bytes.  256 threads.
__device__ __forceinline__ void class_ffn_block(const ClassArgs& c, int64_t j, unsigned char* lds) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lrow = lane & 31, lh = lane >> 5;
    const int D = c.D, H = c.H;
    const int64_t blk = j / c.nparts;
    const int p = static_cast<int>(j - blk * c.nparts);
    bf16_bits* zs = reinterpret_cast<bf16_bits*>(lds);
    float* bs = reinterpret_cast<float*>(lds + static_cast<size_t>(kClsRows) * kClsZPitch * 2);
    const int64_t row0 = blk * kClsRows;
    const int nchunks = (H + kClsChunk - 1) / kClsChunk;
    const int c0 = p * c.per, c1 = c0 + c.per < nchunks ? c0 + c.per : nchunks;

    // Operand offsets: a row past the matrix lies past the buffer resource
    // and reads zeros; a k slot past the row (D or H not a multiple of 16)
    // is sent past it by setting the top bit (arithmetic, not a branch, so
    // that the loads stay straight-line and the waits exact).
    auto oob_if = [](bool past) { return static_cast<uint32_t>(-static_cast<int>(past)) & kRawOob; };
    // W1 operand of chunk hb: wave's hidden row hb + 32 w + l%32, inputs
    // 16 i + 8 (l/32) .. + 8
    const __amdgpu_buffer_rsrc_t w1 = raw_rsrc(c.W1, static_cast<int64_t>(H) * D * 2);
    uint4 a1[kClsKSteps];
    auto load_w1 = [&](int hb) {
        const uint32_t rowoff = static_cast<uint32_t>((hb + 32 * wave + lrow) * D) * 2u;
#pragma unroll
        for (int i = 0; i < kClsKSteps; ++i) {
            const int k = 16 * i + 8 * lh;
            a1[i] = raw_load16(w1, (rowoff + static_cast<uint32_t>(k) * 2u) | oob_if(k >= D));
        }
    };
    // W2 operand of chunk hb: output column 96 w + 32 t + l%32, hidden units
    // hb + 16 s + 8 (l/32) .. + 8
    const __amdgpu_buffer_rsrc_t w2 = raw_rsrc(c.W2, static_cast<int64_t>(D) * H * 2);
    uint4 a2[3][8];
    auto load_w2 = [&](int hb) {
#pragma unroll
        for (int t = 0; t < 3; ++t) {
            const uint32_t rowoff = static_cast<uint32_t>((96 * wave + 32 * t + lrow) * H) * 2u;
#pragma unroll
            for (int s = 0; s < 8; ++s) {
                const int h = hb + 16 * s + 8 * lh;
                a2[t][s] = raw_load16(w2, (rowoff + static_cast<uint32_t>(h) * 2u) | oob_if(h >= H));
            }
        }
    };

    // x operand for the whole pass, in registers: class row l%32 (zeros past
    // the class rows), inputs 16 i + 8 (l/32) .. + 8 (zeros past D)
    uint4 xb[kClsKSteps];
    {
        const int64_t row = row0 + lrow;
        const bf16_bits* xr = c.x + (row < c.ncls ? row : 0) * c.stride * D;
#pragma unroll
        for (int i = 0; i < kClsKSteps; ++i) {
            const int k = 16 * i + 8 * lh;
            xb[i] = (row < c.ncls && k < D) ? *reinterpret_cast<const uint4*>(xr + k)
                                            : make_uint4(0u, 0u, 0u, 0u);
        }
    }
    load_w1(c0 * kClsChunk);
    load_w2(c0 * kClsChunk);
    // b1 (read in every chunk's epilogue from LDS: a global load there would
    // wait for the next chunk's W1 loads issued before it)
    const int hpad = class_hpad(H);
    for (int i = tid; i < hpad; i += 256) bs[i] = (c.b1 != nullptr && i < H) ? c.b1[i] : 0.0f;

    f32x16 acc[3];
#pragma unroll
    for (int t = 0; t < 3; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[t][v] = 0.0f;
    class_lds_barrier();   // b1 in LDS

    for (int ch = c0; ch < c1; ++ch) {
        const int hb = ch * kClsChunk;
        // phase 1: z^T tile (lane: class row l%32, hidden 8 (v/4) + 4 (l/32) + v%4)
        f32x16 zt;
#pragma unroll
        for (int v = 0; v < 16; ++v) zt[v] = 0.0f;
#pragma unroll
        for (int i = 0; i < kClsKSteps; ++i)
            zt = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a1[i]),
                                                         __builtin_bit_cast(bf16x8, xb[i]), zt, 0, 0, 0);
        load_w1(hb + kClsChunk);   // past the part's run on its last chunk: never used
        // bias, GELU, bfloat16 (units past H: zero bias and zero W1 rows, and
        // their W2 columns read as zeros, so they add nothing)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int hl = 32 * wave + 8 * g + 4 * lh;
            const float4 bb = *reinterpret_cast<const float4*>(bs + hb + hl);
            const uint2 pk = make_uint2(pack2_bf16(gelu_erf(zt[4 * g] + bb.x), gelu_erf(zt[4 * g + 1] + bb.y)),
                                        pack2_bf16(gelu_erf(zt[4 * g + 2] + bb.z), gelu_erf(zt[4 * g + 3] + bb.w)));
            *reinterpret_cast<uint2*>(zs + lrow * kClsZPitch + hl) = pk;
        }
        class_lds_barrier();
        // phase 2: y^T tiles (lane: class row l%32, column 8 (v/4) + 4 (l/32) + v%4)
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            const uint4 b = *reinterpret_cast<const uint4*>(zs + lrow * kClsZPitch + 16 * s + 8 * lh);
#pragma unroll
            for (int t = 0; t < 3; ++t)
                acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a2[t][s]),
                                                                 __builtin_bit_cast(bf16x8, b), acc[t], 0, 0, 0);
        }
        load_w2(hb + kClsChunk);
        class_lds_barrier();   // z read before the next chunk rewrites it
    }
    // the loads of the chunk after the run are never used: they land before
    // the wave can end
    __builtin_amdgcn_s_waitcnt(0xF70);   // vmcnt(0)

    if (c.nparts > 1) {
        // partial sums in the lane layout: (wave, tile, 4-value group) runs
        // of 64 lanes x 16 bytes
        float* mine = c.part + (blk * c.nparts + p) * kClsPartFloats;
        auto slot = [&](int t, int q) { return ((wave * 3 + t) * 4 + q) * 256 + lane * 4; };
#pragma unroll
        for (int t = 0; t < 3; ++t)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                *reinterpret_cast<float4*>(mine + slot(t, q)) =
                    make_float4(acc[t][4 * q], acc[t][4 * q + 1], acc[t][4 * q + 2], acc[t][4 * q + 3]);
        // every wave's stores are complete at the barrier; thread 0's
        // agent-scope release covers them, the last part's acquire pairs
        // with the other parts' releases
        __syncthreads();
        __shared__ int s_last;
        if (tid == 0) {
            uint64_t* w = c.count + blk;
            uint64_t old = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            uint64_t nv;
            do {   // at most P rounds: every failure is another part's arrival
                nv = (old >> 16) == c.launch ? old + 1 : (c.launch << 16) | 1u;
            } while (!__hip_atomic_compare_exchange_weak(w, &old, nv, __ATOMIC_ACQ_REL, __ATOMIC_RELAXED,
                                                         __HIP_MEMORY_SCOPE_AGENT));
            s_last = static_cast<int>(nv & 0xffffu) == c.nparts;
        }
        __syncthreads();
        if (!s_last) return;
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        const float* all = c.part + blk * c.nparts * kClsPartFloats;
#pragma unroll
        for (int t = 0; t < 3; ++t)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                float4 sum = *reinterpret_cast<const float4*>(all + slot(t, q));
                for (int pp = 1; pp < c.nparts; ++pp) {
                    const float4 v = *reinterpret_cast<const float4*>(all + pp * kClsPartFloats + slot(t, q));
                    sum.x += v.x; sum.y += v.y; sum.z += v.z; sum.w += v.w;
                }
                acc[t][4 * q] = sum.x; acc[t][4 * q + 1] = sum.y;
                acc[t][4 * q + 2] = sum.z; acc[t][4 * q + 3] = sum.w;
            }
    }

    // y rows: + b2, bfloat16, four consecutive columns per 8-byte store
    const int64_t row = row0 + lrow;
    if (row >= c.ncls) return;
    bf16_bits* yr = c.y + row * c.stride * D;
#pragma unroll
    for (int t = 0; t < 3; ++t) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int n = 96 * wave + 32 * t + 8 * g + 4 * lh;
            if (n >= D) continue;
            float v4[4];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) v4[jj] = acc[t][4 * g + jj] + (c.b2 != nullptr ? c.b2[n + jj] : 0.0f);
            *reinterpret_cast<uint2*>(yr + n) = make_uint2(pack2_bf16(v4[0], v4[1]), pack2_bf16(v4[2], v4[3]));
        }
    }
}

// Host side (class_ffn.hip).  class_ffn_plan fills nparts, per, part, count
// and launch for the class rows of c (part and count: workspace regions of
// kClsPartBytes and kClsCountWords words) and returns the workgroup count.
bool class_ffn_supported(int D, int H);
int64_t class_ffn_plan(ClassArgs& c, float* part, uint64_t* count);
hipError_t launch_class_ffn(const ClassArgs& c, hipStream_t st);

}  // namespace clearmoe
