// Fused top-1 CLEAR-MoE FFN in bfloat16 for gfx950: one kernel from x to y.
// The kernel templates (their body is fused_body.inc); fused.hip
// instantiates the one-workgroup-per-tile variants and holds the host side,
// fused_cls.hip the ones with the class rows' dense FFN on extra
// workgroups, fused_split.hip the hidden-split ones.
//
// With k = 1 every row p of the expert order is one token, and the layer is
//     z      = GELU(x W1^T + b1)                        shared fc1 (Eq. 2)
//     [t|u]  = z [Vt ; Q_e]^T, the u columns times the gate
//     y      = [t|u] [US | P_e]^T + b2                  shared basis + residual (Eq. 2,
//                                                        Algorithm 3)
// A workgroup owns up to 64 consecutive rows of one expert's segment and the
// whole hidden width, so neither z nor [t|u] ever goes to HBM:
//   * the 64 gathered x rows are copied to LDS once and stay there;
//   * wave w walks the 64-wide hidden slices w, w + 4, w + 8, ...: for a slice
//     it forms z^T (64 hidden x 64 tokens, four 32x32 MFMA tiles), its W1 rows
//     streamed by DMA into a ring of LDS stages private to the wave (no
//     workgroup barrier in the loop), applies bias, GELU and bf16 rounding, and
//     adds [Vt;Q_e]_slice z^T_slice to its own [t|u]^T held in registers;
//   * the four partial [t|u] are summed in LDS as (w0 + w2) + (w1 + w3)
//     (fixed order, deterministic), the gate is applied, the sum is rounded to
//     bf16, and the last product builds the y rows in LDS and writes each row
//     to its token with 16-byte stores.
//
// Register chaining.  For v_mfma_f32_32x32x16_bf16, lane l holds result
// column l%32, rows 8(v/4) + 4(l/32) + v%4 (v = 0..15), and as a k operand
// supplies k slots 8(l/32) + i (i = 0..7) of row/column l%32.  Tile q (0, 1)
// of the z^T block takes, in row slot s, W1 row
//     hb + 32 q + 16 (s>>4) + 8 ((s>>2)&1) + 4 ((s>>3)&1) + (s&3),
// which makes lane l's result v of tile q the hidden unit
// hb + 32 q + 16 (v/8) + 8 (l/32) + v%8.  Run j = 2q + v/8 of 8 such values
// is then the B operand of an MFMA whose slot 8(l/32) + i is hidden unit
// hb + 16 j + 8 (l/32) + i, and the A operand ([Vt;Q_e] rows) reads those 8
// units: the two lane halves read 32 contiguous bytes of a row.  Phase-1
// products use their own k order (slot 8(l/32) + i of MFMA j is input feature
// 64 g + 32 (l/32) + 8 j + i), matched by the x reads.
//
// Waits.  The W1 DMA is inline asm the compiler does not see; every wave
// issues its loads in a fixed order (stages, then the [Vt;Q_e] loads of a
// slice after its first two stages) and waits with vmcnt values computed from
// that order.  Loads the compiler does see ([Vt;Q_e], b1) are all complete
// whenever it waits for them, so its own counts never hold back a DMA.
#pragma once

#include <type_traits>

#include "class_ffn.h"
#include "kernels.h"

namespace clearmoe {

struct FusedArgs {
    const bf16_bits* x;
    const bf16_bits* W1;
    const float* b1;
    const bf16_bits* US;
    const bf16_bits* Vt;
    const float* b2;
    const bf16_bits* P;
    const bf16_bits* Q;
    const int32_t* perm;
    const int32_t* offsets;
    const int32_t* idx;          // [T] expert of each token (k = 1), with tile_counts:
    const int32_t* tile_counts;  //   the router's histogram [nh][E] of htile-token tiles;
    int htile, nh;               //   non-NULL: the workgroup finds its rows' tokens itself
    const float* gate;
    bf16_bits* y;
    int64_t T;
    int D, H, E, r, q;
    int xch;        // LDS pitch of an x row, 16-byte chunks (odd, >= 8 * kgroups)
    int hpad;       // H rounded up to 4 waves x 64
    int tuch;       // LDS pitch of a bf16 [t|u] row, 16-byte chunks (odd)
    int yp;         // LDS pitch (elements) of a bf16 y row
    int b2_off;     // byte offset of b2 (after b1)
    int b2_chunks;  // 16-byte chunks of the b2 region (a multiple of 64)
    int x_off;      // byte offset of the x rows (after b2)
    int ring_off;   // byte offset of the four waves' W1 rings (after x)
    int epi_off;    // byte offset of the [t|u] partial sums, later the y rows (after b2)
    int tu_off;     // byte offset of the bf16 [t|u] rows (after the sums / y rows)
    int tiles_bound;
    int per_xcd;
    int split;            // S >= 1 workgroups per tile, each on every S-th hidden slice group
    float* part;          // S > 1: [tiles][S][64][32 NFT] float32 partial [t|u] sums
    int32_t* counters;    // S > 1: [tiles] arrivals, zero before the launch
};

// Launch of the hidden-split variant (fused_split.hip) for nft 32-row [t|u]
// tiles.
hipError_t fused_launch_split(const FusedArgs& a, size_t lds, int grid, int nft, hipStream_t st);
struct ClassArgs;
// Launch of the variant with the class rows' workgroups (fused_cls.hip);
// grid counts the tiles' workgroups and the class rows'.
hipError_t fused_launch_cls(const FusedArgs& a, const ClassArgs& c, size_t lds, int grid, int nft,
                            hipStream_t st);

namespace {


constexpr int kFRows = 64;      // rows (tokens) per workgroup
constexpr int kFHid = 64;       // hidden units per wave per step
constexpr int kFXcds = 8;
constexpr int kFMaxSplit = 8;   // workgroups per tile of a small batch (hidden split)
constexpr int kNS = 3;                  // W1 ring stages per wave
constexpr int kStageBytes = 64 * 128;   // 64 W1 rows x 64 inputs (bf16)
constexpr int kCt = 3;                  // y column tiles per wave (4 kCt tiles cover D)
constexpr int kFGroups = 6;             // 64-wide input groups (D <= 384)

__device__ __attribute__((aligned(16))) const uint32_t g_fused_zero[4] = {0u, 0u, 0u, 0u};

typedef __attribute__((address_space(3))) uint32_t lds_word;
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ void lds_dma16(const void* gptr, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                 :
                 : "s"(lds_addr), "v"(gptr)
                 : "memory", "m0");
}

// Raw buffer resources: a load whose offset lies outside [0, bytes) returns
// zero, so tails and absent rows need no pointer selects and no branches.
constexpr uint32_t kOob = 0x80000000u;          // an offset past every buffer here
constexpr int kBufWord3 = 0x00020000;           // raw dword access (CDNA)

// Two floats -> two bf16 (hardware round to nearest even), packed in 32 bits.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    const f32x2 v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

__device__ __forceinline__ f32x16 mfma(const u32x4& a, const u32x4& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                    __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Buffer descriptor words for the inline-asm DMA below (uniform values).
typedef int i32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i32x4 dma_desc(const void* p, int64_t bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(p);
    i32x4 d;
    d.x = __builtin_amdgcn_readfirstlane(static_cast<int>(a & 0xffffffffu));
    d.y = __builtin_amdgcn_readfirstlane(static_cast<int>((a >> 32) & 0xffffu));   // stride 0
    d.z = __builtin_amdgcn_readfirstlane(static_cast<int>(bytes));
    d.w = kBufWord3;
    return d;
}

// 16 bytes per lane, buffer -> LDS at m0 + 16 * lane (zeros outside the
// buffer); waited for like the ring stages.
__device__ __forceinline__ void dma16_buf(const i32x4& d, uint32_t off, uint32_t m0) {
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :
                 : "s"(m0), "v"(off), "s"(d)
                 : "memory", "m0");
}

// 16 bytes per lane, buffer -> registers (zeros outside the buffer).  Inline
// asm like the DMA: the compiler does not count it, so its own waits never
// drain the W1 stages issued after it.  The caller waits with vm_wait and
// then passes the registers through reg_ready before any use.
// The zero scalar offset sits in a register (not the inline constant), which
// also tells these loads apart from the compiler's in the kernel's ISA.
__device__ __forceinline__ u32x4 bload16_asm(const i32x4& d, uint32_t off, int zero) {
    u32x4 v;
    asm volatile("buffer_load_dwordx4 %0, %1, %2, %3 offen" : "=v"(v) : "v"(off), "s"(d), "s"(zero));
    return v;
}
// After the wait that covers an asm load: uses of v stay below this point.
__device__ __forceinline__ void reg_ready(u32x4& v) { asm volatile("" : "+v"(v)); }

// One W1 ring stage: 8 loads of 16 bytes per lane, buffer -> LDS at
// base + 1024 i + 16 * lane (zeros for an offset outside the buffer).  Inline
// asm: the compiler does not count these loads; the kernel waits for them
// with explicit vmcnt values (vm_wait below).  M0 carries the LDS address; one
// wait state separates each M0 write from the load that reads it.
__device__ __forceinline__ void dma_stage8(const i32x4& d, uint32_t base, const uint32_t (&o)[8]) {
    asm volatile(
        "s_mov_b32 m0, %0\n\ts_nop 0\n\t"
        "buffer_load_dwordx4 %1, %9, 0 offen lds\n\t"
        "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\t"
        "buffer_load_dwordx4 %2, %9, 0 offen lds\n\t"
        "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\t"
        "buffer_load_dwordx4 %3, %9, 0 offen lds\n\t"
        "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\t"
        "buffer_load_dwordx4 %4, %9, 0 offen lds\n\t"
        "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\t"
        "buffer_load_dwordx4 %5, %9, 0 offen lds\n\t"
        "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\t"
        "buffer_load_dwordx4 %6, %9, 0 offen lds\n\t"
        "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\t"
        "buffer_load_dwordx4 %7, %9, 0 offen lds\n\t"
        "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\t"
        "buffer_load_dwordx4 %8, %9, 0 offen lds"
        :
        : "s"(base), "v"(o[0]), "v"(o[1]), "v"(o[2]), "v"(o[3]), "v"(o[4]), "v"(o[5]), "v"(o[6]),
          "v"(o[7]), "s"(d)
        : "memory", "m0", "scc");
}

// Wait until at most N vector-memory loads of this wave are outstanding.  The
// memory clobber keeps LDS reads of the awaited data below it.
template <int N>
__device__ __forceinline__ void vm_wait() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

__device__ __forceinline__ int swz(int row) { return (row >> 1) & 7; }

// Hidden offset (within a 64-slice) of row slot s of z^T tile q.  It makes
// the lane's result v of tile q (row slot 8(v/4) + 4 lh + v%4) the hidden
// unit 32 q + 16 (v/8) + 8 lh + v%8.
__device__ __forceinline__ int hid_of_slot(int q, int s) {
    return 32 * q + 16 * (s >> 4) + 8 * ((s >> 2) & 1) + 4 * ((s >> 3) & 1) + (s & 3);
}


// [Vt;Q_e] halves (issued in steps 4 and 5 of every block, before that step's
// W1 stage) issued after stage n was: stage n of step g was issued in step
// g - 2, of the previous block when negative (the first block has none; its
// stages 0 and 1 come from the prologue).
__host__ __device__ constexpr int vq_halves_after(int g, int kgroups, bool first) {
    const int s = g - 2;
    int c = 0;
    for (int p = 4; p <= 5; ++p) {
        if (s >= 0) c += (p > s && p <= g) ? 1 : 0;
        else c += ((!first && p > kgroups + s) || p <= g) ? 1 : 0;
    }
    return c;
}
static_assert(vq_halves_after(0, 6, false) == 1 && vq_halves_after(1, 6, false) == 0 &&
                  vq_halves_after(0, 6, true) == 0 && vq_halves_after(4, 6, false) == 1 &&
                  vq_halves_after(5, 6, false) == 2 && vq_halves_after(0, 8, false) == 0 &&
                  vq_halves_after(6, 8, false) == 1 && vq_halves_after(5, 6, true) == 2,
              "vq issue accounting");

// Bare workgroup barrier: LDS operations complete, outstanding DMA untouched
// (__syncthreads would also wait for every vector-memory load).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
}

// Inclusive prefix sum over the 64 lanes of a wave by DPP: shifts by 1, 2, 4
// and 8 lanes within rows of 16 (lanes without a source add 0), then lane 15
// of each row into the next row and lane 31 into rows 2 and 3.
__device__ __forceinline__ int wave_incl_scan(int v) {
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);   // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);   // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);   // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);   // row_shr:8
    v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);   // row_bcast:15
    v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);   // row_bcast:31
    return v;
}

// NFT = 32-row tiles of [t|u] features (r + q <= 32 NFT).  The number of
// 64-wide input groups is kFGroups (D <= 384, padded groups read zeros), so
// phase 1 is straight-line code.
template <int NFT, bool SPLIT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_fused_top1(FusedArgs a) {
#include "fused_body.inc"
}

// The one-workgroup-per-tile kernel with the class rows' dense FFN
// (class_ffn.h) on the workgroups past the tiles: they start with the tiles,
// on the CUs the tiles leave free, and need no launch of their own.
template <int NFT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_fused_top1_cls(FusedArgs a, ClassArgs c) {
    if (static_cast<int>(blockIdx.x) >= a.per_xcd * kFXcds) {
        extern __shared__ __attribute__((aligned(1024))) unsigned char cls_smem[];
        class_ffn_block(c, static_cast<int>(blockIdx.x) - a.per_xcd * kFXcds, cls_smem);
        return;
    }
    constexpr bool SPLIT = false;
#include "fused_body.inc"
}

template <int NFT, bool SPLIT>
hipError_t fused_cfg(const FusedArgs& a, size_t lds, int grid, hipStream_t st) {
    if (lds > 65536) {
        const hipError_t err = hipFuncSetAttribute(
            reinterpret_cast<const void*>(&k_fused_top1<NFT, SPLIT>),
            hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(lds));
        if (err != hipSuccess) return err;
    }
    launch_kernel(k_fused_top1<NFT, SPLIT>, dim3(static_cast<unsigned>(grid)), 256, lds, st, a);
    return hipGetLastError();
}

template <int NFT>
hipError_t fused_cfg_cls(const FusedArgs& a, const ClassArgs& c, size_t lds, int grid, hipStream_t st) {
    if (lds > 65536) {
        const hipError_t err = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_fused_top1_cls<NFT>),
                                                   hipFuncAttributeMaxDynamicSharedMemorySize,
                                                   static_cast<int>(lds));
        if (err != hipSuccess) return err;
    }
    launch_kernel(k_fused_top1_cls<NFT>, dim3(static_cast<unsigned>(grid)), 256, lds, st, a, c);
    return hipGetLastError();
}

}  // namespace

}  // namespace clearmoe
