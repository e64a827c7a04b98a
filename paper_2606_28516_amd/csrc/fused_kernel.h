// Fused top-1 CLEAR-MoE FFN in bfloat16 for gfx950: one kernel from x to y.
// The kernel template; fused.hip instantiates the one-workgroup-per-tile
// variants and holds the host side, fused_split.hip the hidden-split ones.
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
    extern __shared__ __attribute__((aligned(1024))) unsigned char smem[];
    __shared__ int32_t s_tok[kFRows];
    __shared__ float s_gate[kFRows];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lrow = lane & 31, lh = lane >> 5;

    // ---- tile -> (expert e, rows [m_lo, m_hi)), XCD-major order
    const int wg = (blockIdx.x % kFXcds) * a.per_xcd + blockIdx.x / kFXcds;
    const int tile = SPLIT ? wg / a.split : wg, part = SPLIT ? wg - tile * a.split : 0;
    if (tile >= a.tiles_bound) return;
    const int D = a.D, H = a.H, r = a.r, rq = a.r + a.q;

    float* s_b1 = reinterpret_cast<float*>(smem);
    const float* s_b2 = reinterpret_cast<const float*>(smem + a.b2_off);
    const unsigned char* xs = smem + a.x_off;
    unsigned char* ringp = smem + a.ring_off + wave * (kNS * kStageBytes);
    const uint32_t ring = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_word*)ringp));
    constexpr int kgroups = kFGroups;
    // hidden slices of this wave: slot, slot + 4 S, ... (slot = 4 part + wave)
    const int slot = SPLIT ? 4 * part + wave : wave, nslot = SPLIT ? 4 * a.split : 4;
    const int n_iter = slot * kFHid < H ? (H - slot * kFHid + nslot * kFHid - 1) / (nslot * kFHid) : 0;
    const i32x4 d_w1 = dma_desc(a.W1, static_cast<int64_t>(H) * D * 2);

    // DMA of W1 ring stage n = slice it, input group g into slot n % kNS: ring
    // row 32q + s holds W1 row hb + hid_of_slot(q, s), and its 16-byte chunk c
    // (inputs 64g + 8c .. + 8) sits at slot c ^ swz(row).
    auto dma_stage = [&](int n) {
        const int it = n / kgroups, g = n - it * kgroups;
        const int hb = (it * nslot + slot) * kFHid;
        const uint32_t m0 = ring + static_cast<uint32_t>(n % kNS) * kStageBytes;
        uint32_t off[8];
#pragma unroll
        for (int ins = 0; ins < 8; ++ins) {
            const int row = 8 * ins + (lane >> 3);
            const int c = (lane & 7) ^ swz(row);
            const int hid = hb + hid_of_slot(row >> 5, row & 31);
            const int k = 64 * g + 8 * c;
            off[ins] = ((hid < H) & (k < D)) ? static_cast<uint32_t>(hid * D + k) * 2u : kOob;
        }
        // the slot's previous stage must have been read by this wave
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        dma_stage8(d_w1, __builtin_amdgcn_readfirstlane(m0), off);
    };

    // ---- b1, b2 and the first two W1 stages -> LDS by DMA, issued before the
    //      tile's tokens are known (they do not depend on them); early exits
    //      below wait for them first
    {
        const uint32_t lb = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_word*)smem));
        const i32x4 d_b1 = dma_desc(a.b1, a.b1 != nullptr ? static_cast<int64_t>(H) * 4 : 0);
        const i32x4 d_b2 = dma_desc(a.b2, a.b2 != nullptr ? static_cast<int64_t>(D) * 4 : 0);
        for (int base = wave * 64; base < a.hpad / 4; base += 256)    // zeros past H
            dma16_buf(d_b1, static_cast<uint32_t>(base + lane) * 16u,
                      __builtin_amdgcn_readfirstlane(lb + base * 16));
        for (int base = wave * 64; base < a.b2_chunks; base += 256)   // zeros past D
            dma16_buf(d_b2, static_cast<uint32_t>(base + lane) * 16u,
                      __builtin_amdgcn_readfirstlane(lb + a.b2_off + base * 16));
    }
    if (n_iter > 0) {
        dma_stage(0);
        dma_stage(1);
    }

    const bool own_dispatch = a.tile_counts != nullptr;
    __shared__ int s_off[64];                   // expert totals (own dispatch)
    __shared__ int s_nlist;
    if (own_dispatch) {
        // Expert totals from the router's histogram (staged in the x region,
        // free until the gather): thread tid sums expert tid % E over tiles
        // tid / E + G i, then one LDS atomic; thread 0 scans them.
        int* s_h = reinterpret_cast<int*>(smem + a.x_off);
        const int nhE = a.nh * a.E;
        for (int i = tid; i < nhE; i += 256) s_h[i] = a.tile_counts[i];
        if (tid < a.E) s_off[tid] = 0;
        if (tid == 0) s_nlist = 0;
        __syncthreads();
        const int G = 256 / a.E;
        if (tid < G * a.E) {
            const int ee = tid % a.E;
            int c = 0;
            for (int b = tid / a.E; b < a.nh; b += G) c += s_h[b * a.E + ee];
            atomicAdd(&s_off[ee], c);
        }
        __syncthreads();
    }
    int e = -1;
    int64_t m_lo = 0, m_hi = 0;
    int e_lo = 0;                               // first row of expert e
    if (own_dispatch) {
        // every wave alike: lane s < E holds expert s's total; prefix sums
        // over the lanes give its rows and its tiles, and the first lane
        // whose tiles end past this tile is the expert
        const int M = static_cast<int>(a.T);
        int tot = lane < a.E ? s_off[lane] : 0;
        tot = tot < 0 ? 0 : (tot > M ? M : tot);
        int hi = wave_incl_scan(tot);
        hi = hi > M ? M : hi;
        const int lo = (hi - tot) > M ? M : (hi - tot);
        const int nt = (hi - lo + kFRows - 1) / kFRows;
        const int tend = wave_incl_scan(nt);
        const uint64_t hit = __ballot(lane < a.E && tile < tend);
        if (hit != 0) {
            e = __builtin_ctzll(hit);
            e_lo = __builtin_amdgcn_readlane(lo, e);
            const int e_hi = __builtin_amdgcn_readlane(hi, e);
            const int t0 = __builtin_amdgcn_readlane(tend - nt, e);
            m_lo = e_lo + static_cast<int64_t>(tile - t0) * kFRows;
            m_hi = m_lo + kFRows < e_hi ? m_lo + kFRows : e_hi;
        }
    } else {
        const int64_t M = a.T;
        int64_t before = 0;
        for (int s = 0; s < a.E; ++s) {
            // offsets are clamped to [0, T]: bad offsets cannot send a
            // workgroup outside the buffers
            // read as uniform values (the same for every lane), so that e
            // and the expert's buffer descriptors below live in scalar registers
            int64_t lo = __builtin_amdgcn_readfirstlane(a.offsets[s]);
            int64_t hi = __builtin_amdgcn_readfirstlane(a.offsets[s + 1]);
            lo = lo < 0 ? 0 : (lo > M ? M : lo);
            hi = hi < lo ? lo : (hi > M ? M : hi);
            const int64_t nt = (hi - lo + kFRows - 1) / kFRows;
            if (tile < before + nt) {
                e = s;
                m_lo = lo + (tile - before) * kFRows;
                m_hi = m_lo + kFRows < hi ? m_lo + kFRows : hi;
                break;
            }
            before += nt;
        }
    }
    if (e < 0) {                                // uniform over the workgroup
        vm_wait<0>();
        return;
    }
    const int rows = static_cast<int>(m_hi - m_lo);

    if (own_dispatch) {
        // The tokens of ranks [rlo, rhi) of expert e in the stable order (by
        // token index).  A block scan over the histogram column of e gives
        // every tile's first rank; the tiles that hold ranks of the range (at
        // most 64: each holds at least one) go to a list, and the waves scan
        // their idx with ballots, each rank's token landing in s_tok.
        const int* s_h = reinterpret_cast<const int*>(smem + a.x_off);
        int2* s_list = reinterpret_cast<int2*>(smem + a.x_off) + (a.nh * a.E + 1) / 2;
        __shared__ int s_wsum[4];
        const int rlo = static_cast<int>(m_lo) - e_lo, rhi = static_cast<int>(m_hi) - e_lo;
        const int per = (a.nh + 255) / 256;
        const int b0 = tid * per, b1 = b0 + per < a.nh ? b0 + per : a.nh;
        int mine = 0;
        for (int b = b0; b < b1; ++b) mine += s_h[b * a.E + e];
        const int incl = wave_incl_scan(mine);  // inclusive scan over the block
        if (lane == 63) s_wsum[wave] = incl;
        if (tid < kFRows) s_tok[tid] = -1;
        __syncthreads();
        int pre = incl - mine;
        for (int i = 0; i < wave; ++i) pre += s_wsum[i];
        for (int b = b0; b < b1; ++b) {
            const int c = s_h[b * a.E + e];
            if (c > 0 && pre < rhi && pre + c > rlo) {
                const int at = atomicAdd(&s_nlist, 1);
                if (at < kFRows) s_list[at] = make_int2(b, pre);
            }
            pre += c;
        }
        __syncthreads();
        const int nlist = s_nlist < kFRows ? s_nlist : kFRows;
        const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
        // a wave's 64-token chunks of its listed tiles, up to 8 loads in
        // flight before the ballots use them
        const int cpt = a.htile / 64;                  // chunks per tile
        for (int li0 = wave; li0 < nlist; li0 += 4 * (8 / cpt)) {
            int exv[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int li = li0 + 4 * (j / cpt);
                const int c0 = 64 * (j % cpt);
                exv[j] = -1;
                if (li < nlist && j < 8 / cpt * cpt) {
                    const int64_t t = static_cast<int64_t>(s_list[li].x) * a.htile + c0 + lane;
                    if (t < a.T) exv[j] = a.idx[t];
                }
            }
            int run = 0;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int li = li0 + 4 * (j / cpt);
                if (li >= nlist || j >= 8 / cpt * cpt) break;   // uniform
                const int c0 = 64 * (j % cpt);
                if (c0 == 0) run = s_list[li].y;
                const uint64_t m = __ballot(exv[j] == e);
                const int rank = run + __popcll(m & below);
                const int64_t t = static_cast<int64_t>(s_list[li].x) * a.htile + c0 + lane;
                if (exv[j] == e && rank >= rlo && rank < rhi) s_tok[rank - rlo] = static_cast<int32_t>(t);
                run += __popcll(m);
            }
        }
        __syncthreads();
        // top-1 gates are exactly 1 (the softmax of one selected logit)
        if (tid < kFRows) {
            const int32_t t = s_tok[tid];
            const bool ok = tid < rows && t >= 0 && t < a.T;
            s_gate[tid] = ok ? 1.0f : 0.0f;
            if (!ok) s_tok[tid] = -1;
        }
    } else if (tid < kFRows) {
        int32_t tok = -1;
        float g = 0.0f;
        if (tid < rows) {
            const int32_t t = a.perm[m_lo + tid];
            if (t >= 0 && t < a.T) {
                tok = t;
                g = a.gate[t];
            }
        }
        s_tok[tid] = tok;
        s_gate[tid] = g;
    }
    __syncthreads();

    {
        const uint32_t xl = static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lds_word*)xs));
        const int dch = D / 8;
        const int slots = kFRows * a.xch;
        for (int base = wave * 64; base < slots; base += 256) {
            const int j = base + lane;
            const int row = j / a.xch, c = j - row * a.xch;
            const void* src = g_fused_zero;                 // padding chunks read zeros
            if (j < slots && c < dch) {
                const int32_t tok = s_tok[row];
                if (tok >= 0) src = a.x + static_cast<int64_t>(tok) * D + 8 * c;
            }
            lds_dma16(src, __builtin_amdgcn_readfirstlane(xl + base * 16));
        }
    }
    vm_wait<0>();                                      // b1, b2, x and the first stages
    lds_barrier();

    // [Vt;Q_e] are loaded by asm, like the W1 stages, so that the compiler's
    // own waits never drain the stages issued after them; the wave's explicit
    // waits cover them (the step loop is straight-line, so no loop-carried
    // copy of a register can be read before its load lands).
    const int soff0 = __builtin_amdgcn_readfirstlane(static_cast<int>(a.T >> 62));   // 0
    const i32x4 d_vt = dma_desc(a.Vt, static_cast<int64_t>(r) * H * 2);
    const i32x4 d_qe = dma_desc(a.Q + static_cast<int64_t>(e) * a.q * H, static_cast<int64_t>(a.q) * H * 2);
    // LDS byte offsets of this lane's x chunks for token blocks 0 and 1
    const int xoff0 = (lrow * a.xch + 4 * lh) * 16;
    const int xoff1 = xoff0 + 32 * a.xch * 16;

    f32x16 tu[NFT][2];
#pragma unroll
    for (int f = 0; f < NFT; ++f)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int v = 0; v < 16; ++v) tu[f][b][v] = 0.0f;

    // Software pipeline over this wave's slices.  Block k runs phase 1 of
    // slice k (z^T accumulated in za, one ring stage per step) and, in its
    // first four steps, GELU + phase 2 of slice k - 1 (one run j of 8 hidden
    // units per step, from zp), so that the GELU arithmetic overlaps the MFMA
    // and LDS work of phase 1.  The [Vt;Q_e] operands of slice k are loaded in
    // step 4 of block k, after the last run of slice k - 1 has used vq.
    f32x16 za[2][2], zp[2][2];
    u32x4 vq[NFT][4];

    // [Vt;Q_e] columns hb + 16 j + 8 lh + [0, 8) for j in [j0, j0 + 2)
    auto load_vq = [&](int hb, int j0) {
#pragma unroll
        for (int f = 0; f < NFT; ++f) {
            // r is a multiple of 32: a feature tile is all Vt rows or all Q_e rows
            const bool tile_vt = 32 * f < r;
            const int feat = 32 * f + lrow;
            const uint32_t rowb = static_cast<uint32_t>(tile_vt ? feat : feat - r) * H * 2;
            const bool live = feat < rq;
#pragma unroll
            for (int jj = 0; jj < 2; ++jj) {
                const int j = j0 + jj;
                const int hid = hb + 16 * j + 8 * lh;
                const uint32_t off = (live & (hid < H)) ? rowb + 2u * hid : kOob;
                vq[f][j] = bload16_asm(tile_vt ? d_vt : d_qe, off, soff0);
            }
        }
    };
    // Run j of the pending slice (hidden units hb + 16 j + 8 lh + i): GELU and
    // bf16 turn the lane's z values (bias included) into the B operand zo, and
    // [t|u]^T += [Vt;Q_e]_run z^T_run.  Units >= H have zero [Vt;Q_e] columns.
    auto gelu_run = [&](int j, u32x4 (&zo)[2]) {
        const int qq = j >> 1, v0 = 8 * (j & 1);
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int v = v0 + 2 * i;
                zo[b][i] = pack_bf16x2(gelu_erf(zp[qq][b][v]), gelu_erf(zp[qq][b][v + 1]));
            }
    };
    auto phase2_run = [&](int j, const u32x4 (&zo)[2]) {
#pragma unroll
        for (int f = 0; f < NFT; ++f)
#pragma unroll
            for (int b = 0; b < 2; ++b) tu[f][b] = mfma(vq[f][j], zo[b], tu[f][b]);
    };
    // Phase-1 step: stage n of the ring (inputs 64 g .. 64 g + 63).
    auto step = [&](int n, int g) {
        const unsigned char* st = ringp + (n % kNS) * kStageBytes;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int c = (8 * g + j) * 16;
            const u32x4 x0 = *reinterpret_cast<const u32x4*>(xs + xoff0 + c);
            const u32x4 x1 = *reinterpret_cast<const u32x4*>(xs + xoff1 + c);
#pragma unroll
            for (int qq = 0; qq < 2; ++qq) {
                const int row = 32 * qq + lrow;
                const u32x4 w = *reinterpret_cast<const u32x4*>(
                    st + row * 128 + (((4 * lh + j) ^ swz(row)) << 4));
                za[qq][0] = mfma(w, x0, za[qq][0]);
                za[qq][1] = mfma(w, x1, za[qq][1]);
            }
        }
    };
    // Block k.  In steps 0..3 the GELU of run g of slice k - 1 is computed and
    // the [t|u] MFMAs of run g - 1 are issued (one step later, so that a step
    // holds 26 independent MFMAs next to its GELU arithmetic); run 3's MFMAs
    // come in step 4, before step 5 reloads vq's second half.
    // Loads issued after stage n: stages n + 1 and n + 2 (16), plus
    // the halves of [Vt;Q_e] (2 NFT loads each, issued in steps 4 and 5 before
    // that step's stage) that came after stage n.  The stages past the last
    // slice load zeros (every block issues the same loads).
    // P2 (compile time) keeps a step's phase-1 and GELU work in one basic
    // block, where the scheduler can interleave them.
    auto block = [&](int k, auto p2_tag) {
        constexpr bool p2 = decltype(p2_tag)::value;
        const int hb = (k * nslot + slot) * kFHid;
        // z^T accumulators start at b1 (lane's value v of tile qq is hidden
        // unit hb + 32 qq + 16 (v/8) + 8 lh + v%8; the LDS copy of b1 is zero
        // past H)
#pragma unroll
        for (int qq = 0; qq < 2; ++qq) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float4 bv = *reinterpret_cast<const float4*>(
                    s_b1 + hb + 32 * qq + 16 * (i >> 1) + 8 * lh + 4 * (i & 1));
#pragma unroll
                for (int b = 0; b < 2; ++b) {
                    za[qq][b][4 * i] = bv.x;
                    za[qq][b][4 * i + 1] = bv.y;
                    za[qq][b][4 * i + 2] = bv.z;
                    za[qq][b][4 * i + 3] = bv.w;
                }
            }
        }
        u32x4 zo_prev[2], zo_cur[2];
#pragma unroll
        for (int g = 0; g < kgroups; ++g) {
            const int n = k * kgroups + g;
            if (g == 4) load_vq(hb, 0);
            if (g == 5) load_vq(hb, 2);
            dma_stage(n + 2);
            switch (vq_halves_after(g, kgroups, !p2)) {
                case 0: vm_wait<16>(); break;
                case 1: vm_wait<16 + 2 * NFT>(); break;
                default: vm_wait<16 + 4 * NFT>(); break;
            }
            if constexpr (p2) {
                // this wait covers stage n, issued in step 5 of the previous
                // block after that block's [Vt;Q_e] loads: vq has landed
                if (g == 1) {
#pragma unroll
                    for (int f = 0; f < NFT; ++f)
#pragma unroll
                        for (int j = 0; j < 4; ++j) reg_ready(vq[f][j]);
                }
            }
            step(n, g);
            if constexpr (p2) {
                if (g >= 1 && g <= 4) phase2_run(g - 1, zo_prev);
                if (g < 4) {
                    gelu_run(g, zo_cur);
#pragma unroll
                    for (int b = 0; b < 2; ++b) zo_prev[b] = zo_cur[b];
                    // spread this step's MFMAs (16, plus 10 from g >= 1) evenly
                    // over its GELU arithmetic, so the matrix pipe never idles
#pragma unroll
                    for (int i = 0; i < 26; ++i) {
                        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);    // one MFMA
                        __builtin_amdgcn_sched_group_barrier(0x002, 12, 0);   // twelve VALU
                    }
                }
            }
        }
#pragma unroll
        for (int qq = 0; qq < 2; ++qq)
#pragma unroll
            for (int b = 0; b < 2; ++b) zp[qq][b] = za[qq][b];
    };

    if (n_iter > 0) {
        block(0, std::false_type{});
        for (int k = 1; k < n_iter; ++k) block(k, std::true_type{});
        // drain: GELU + phase 2 of the last slice, once its [Vt;Q_e] landed
        vm_wait<0>();
#pragma unroll
        for (int f = 0; f < NFT; ++f)
#pragma unroll
            for (int j = 0; j < 4; ++j) reg_ready(vq[f][j]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            u32x4 zo[2];
            gelu_run(j, zo);
            phase2_run(j, zo);
        }
    }
    vm_wait<0>();

    // [US | P_e] operands of this wave's output columns (tiles wave + 4 c; the
    // host admits D <= 128 kCt, so one pass covers every column), issued now
    // by asm so that they stay here and their latency hides behind the
    // reduction.  A k step is all US columns or all P_e columns (r is a
    // multiple of 16); columns past r + q and rows past D read zeros.
    const i32x4 d_us = dma_desc(a.US, static_cast<int64_t>(D) * r * 2);
    const i32x4 d_pe = dma_desc(a.P + static_cast<int64_t>(e) * D * a.q, static_cast<int64_t>(D) * a.q * 2);
    u32x4 bw[kCt][2 * NFT];
#pragma unroll
    for (int c = 0; c < kCt; ++c) {
        const int n = 32 * (wave + 4 * c) + lrow;
#pragma unroll
        for (int ks = 0; ks < 2 * NFT; ++ks) {
            const int k = 16 * ks + 8 * lh;
            const bool step_us = 16 * ks < r;
            const uint32_t off = step_us ? static_cast<uint32_t>(n * r + k) * 2
                                         : static_cast<uint32_t>(n * a.q + k - r) * 2;
            bw[c][ks] = bload16_asm(step_us ? d_us : d_pe, ((n < D) & (k < rq)) ? off : kOob, soff0);
        }
    }

    // ---- sum the four waves' [t|u]^T partials, in two rounds of feature
    //      tiles ([0, kRa) and [kRa, NFT)).  Each wave stores its partial
    //      tiles as [token][feature] floats (16-byte moves; pitch 32 n + 4
    //      floats puts 16 tokens' moves in 16 different bank groups), then
    //      sums 16 tokens of all four as (w0 + w2) + (w1 + w3) (fixed order,
    //      deterministic), gates the u features, rounds to bf16 and writes
    //      the token's row of tul.
    constexpr int kRa = (NFT + 1) / 2;
    lds_barrier();                                     // x and the rings no longer read
    float* areas = reinterpret_cast<float*>(smem + a.epi_off);
    bf16_bits* tul = reinterpret_cast<bf16_bits*>(smem + a.tu_off);
    // hidden split (S > 1): a part's four-wave sums go to its slot of the
    // partial buffer instead (float32, [tile][part][token][32 NFT]), written
    // and read with device-scope (sc1) accesses: they miss the CU's L1 and are
    // coherent across the XCDs' L2s, as relaxed device-scope atomics are
    constexpr bool split = SPLIT;
    constexpr int kFP = 32 * NFT;
    constexpr int kDevScope = 16;    // cache-policy bits: sc1
    const __amdgpu_buffer_rsrc_t tpart = __builtin_amdgcn_make_buffer_rsrc(
        split ? a.part + static_cast<int64_t>(tile) * a.split * kFRows * kFP : nullptr, 0,
        split ? a.split * kFRows * kFP * 4 : 0, kBufWord3);
    auto round = [&](auto f0_tag, auto nt_tag) {
        constexpr int f0 = decltype(f0_tag)::value, nt = decltype(nt_tag)::value;
        constexpr int rp = 32 * nt + 4;
        float* mine = areas + wave * (kFRows * rp);
#pragma unroll
        for (int f = f0; f < f0 + nt; ++f)
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    float4 v;
                    v.x = tu[f][b][4 * g]; v.y = tu[f][b][4 * g + 1];
                    v.z = tu[f][b][4 * g + 2]; v.w = tu[f][b][4 * g + 3];
                    *reinterpret_cast<float4*>(mine + (32 * b + lrow) * rp + 32 * (f - f0) + 8 * g + 4 * lh) = v;
                }
        lds_barrier();
        // lane: token 16 wave + (lane & 15), 4-feature chunks (lane >> 4) + 4 i
        const int t = 16 * wave + (lane & 15);
        const float gt = s_gate[t];
#pragma unroll
        for (int i = 0; i < 2 * nt; ++i) {
            const int c4 = (lane >> 4) + 4 * i;
            float4 o[4];
#pragma unroll
            for (int w = 0; w < 4; ++w)
                o[w] = *reinterpret_cast<const float4*>(areas + w * (kFRows * rp) + t * rp + 4 * c4);
            const int feat = 32 * f0 + 4 * c4;
            float4 sum;
            sum.x = (o[0].x + o[2].x) + (o[1].x + o[3].x);
            sum.y = (o[0].y + o[2].y) + (o[1].y + o[3].y);
            sum.z = (o[0].z + o[2].z) + (o[1].z + o[3].z);
            sum.w = (o[0].w + o[2].w) + (o[1].w + o[3].w);
            if constexpr (split) {
                f32x4 v = {sum.x, sum.y, sum.z, sum.w};
                __builtin_amdgcn_raw_buffer_store_b128(v, tpart, ((part * kFRows + t) * kFP + feat) * 4,
                                                       0, kDevScope);
            } else {
                const float sc = feat < r ? 1.0f : gt;
                uint2 wv;
                wv.x = pack_bf16x2(sum.x * sc, sum.y * sc);
                wv.y = pack_bf16x2(sum.z * sc, sum.w * sc);
                *reinterpret_cast<uint2*>(tul + t * a.tuch * 8 + feat) = wv;
            }
        }
        lds_barrier();
    };
    round(std::integral_constant<int, 0>{}, std::integral_constant<int, kRa>{});
    if constexpr (NFT > kRa)
        round(std::integral_constant<int, kRa>{}, std::integral_constant<int, NFT - kRa>{});
    if constexpr (split) {
        // publish this part's sums: its stores have completed at device scope
        // before the tile's arrival counter is bumped; the last part of the
        // tile to arrive loads all S only after it has seen the count, and
        // sums them in part order (deterministic whatever the arrival order),
        // gates the u features, rounds to bf16 and finishes the tile.  (An
        // agent-scope fence here is an L2 write-back and invalidate on each
        // XCD: 15-35 % slower at 1568-6304 tokens.)
        __shared__ int s_last;
        vm_wait<0>();
        __syncthreads();
        if (tid == 0)
            s_last = __hip_atomic_fetch_add(a.counters + tile, 1, __ATOMIC_RELAXED,
                                            __HIP_MEMORY_SCOPE_AGENT) == a.split - 1;
        __syncthreads();
        if (!s_last) {
            vm_wait<0>();                              // the [US|P_e] loads above
            return;
        }
        const int S = a.split;
        for (int item = tid; item < kFRows * (kFP / 4); item += 256) {
            const int t = item / (kFP / 4), c4 = item - t * (kFP / 4);
            f32x4 v[kFMaxSplit];
#pragma unroll
            for (int pp = 0; pp < kFMaxSplit; ++pp)
                if (pp < S)
                    v[pp] = __builtin_amdgcn_raw_buffer_load_b128(
                        tpart, ((pp * kFRows + t) * kFP + 4 * c4) * 4, 0, kDevScope);
            f32x4 sum = v[0];
#pragma unroll
            for (int pp = 1; pp < kFMaxSplit; ++pp)
                if (pp < S) {
                    sum.x += v[pp].x;
                    sum.y += v[pp].y;
                    sum.z += v[pp].z;
                    sum.w += v[pp].w;
                }
            const int feat = 4 * c4;
            const float sc = feat < r ? 1.0f : s_gate[t];
            uint2 wv;
            wv.x = pack_bf16x2(sum.x * sc, sum.y * sc);
            wv.y = pack_bf16x2(sum.z * sc, sum.w * sc);
            *reinterpret_cast<uint2*>(tul + t * a.tuch * 8 + feat) = wv;
        }
        lds_barrier();
    }

    // ---- y = [t|u] [US | P_e]^T + b2 into LDS rows (over the sums' area,
    //      free now): y^T[n][token] = [US|P_e][n][k] [t|u]^T[k][token]; the
    //      lane holds, for token 32 b + lrow, columns 32 ct + 8 g + 4 lh + [0, 4)
    //      of v-group g.  Features past r + q are zeros on both sides.
    vm_wait<0>();
#pragma unroll
    for (int c = 0; c < kCt; ++c)
#pragma unroll
        for (int ks = 0; ks < 2 * NFT; ++ks) reg_ready(bw[c][ks]);
    bf16_bits* yl = reinterpret_cast<bf16_bits*>(smem + a.epi_off);
    {
        f32x16 ay[kCt][2];
#pragma unroll
        for (int c = 0; c < kCt; ++c)
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int v = 0; v < 16; ++v) ay[c][b][v] = 0.0f;
#pragma unroll
        for (int ks = 0; ks < 2 * NFT; ++ks) {
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const u32x4 tv = *reinterpret_cast<const u32x4*>(
                    tul + ((32 * b + lrow) * a.tuch + 2 * ks + lh) * 8);
#pragma unroll
                for (int c = 0; c < kCt; ++c) ay[c][b] = mfma(bw[c][ks], tv, ay[c][b]);
            }
        }
#pragma unroll
        for (int c = 0; c < kCt; ++c) {
            const int ct = wave + 4 * c;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int n0 = 32 * ct + 8 * g + 4 * lh;
                if (n0 < D) {                               // D % 8 == 0: all four or none
                    const float4 bn = *reinterpret_cast<const float4*>(s_b2 + n0);
#pragma unroll
                    for (int b = 0; b < 2; ++b) {
                        uint2 w;
                        w.x = pack_bf16x2(ay[c][b][4 * g] + bn.x, ay[c][b][4 * g + 1] + bn.y);
                        w.y = pack_bf16x2(ay[c][b][4 * g + 2] + bn.z, ay[c][b][4 * g + 3] + bn.w);
                        *reinterpret_cast<uint2*>(yl + (32 * b + lrow) * a.yp + n0) = w;
                    }
                }
            }
        }
    }
    __syncthreads();
    // ---- y rows -> HBM: wave w writes rows w + 4 i (i < 16), lane c the
    //      16-byte chunks c, c + 64, ...: all LDS reads of a pass, then its stores
    const int dch = D / 8;
    for (int c = lane; c - lane < dch; c += 64) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {                  // 8 rows per batch
            u32x4 v[kFRows / 8];
            const int cc = c < dch ? c : 0;             // lanes past the row read chunk 0
#pragma unroll
            for (int i = 0; i < kFRows / 8; ++i)
                v[i] = *reinterpret_cast<const u32x4*>(yl + (wave + 4 * (8 * h + i)) * a.yp + 8 * cc);
#pragma unroll
            for (int i = 0; i < kFRows / 8; ++i) {
                const int32_t tok = s_tok[wave + 4 * (8 * h + i)];
                if (tok >= 0 && c < dch)
                    *reinterpret_cast<u32x4*>(a.y + static_cast<int64_t>(tok) * D + 8 * c) = v[i];
            }
        }
    }
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

}  // namespace

}  // namespace clearmoe
