// Fused top-1 CLEAR-MoE FFN in bfloat16 for gfx950 (kernel in fused_kernel.h):
// host side, LDS plan, the one-workgroup-per-tile instantiations (those with
// the class rows' workgroups: fused_cls.hip), and the choice of the hidden
// split for small batches.
#include "fused_kernel.h"

namespace clearmoe {

namespace {

int odd_at_least(int n) { return n | 1; }

// 64-wide input groups of phase 1: ceil(D / 64), even, and at least 6 (the
// pipeline spreads a slice's four GELU runs over the first four steps and
// loads the next [Vt;Q_e] in step 4; padded groups read zeros).
int fused_kgroups(int D) {
    const int g = (((D + 63) / 64) + 1) & ~1;
    return g < 6 ? 6 : g;
}

constexpr size_t kLdsBytes = 160 * 1024;   // gfx950 LDS per workgroup
constexpr size_t kStaticLds = 1024;        // s_tok, s_gate (aligned)

// LDS plan: [b1 | b2 | x rows | 4 W1 rings] while the hidden loop runs, then
// [b1 | b2 | the four waves' fp32 [t|u] partial sums of one reduction round,
// later the bf16 y rows | bf16 [t|u] rows] (aliasing x and the rings).
struct FusedLds {
    size_t b1, b2, x, ring, areas, yrows, epi_off, tu_off, total;
    int xch, tuch, yp;
};
FusedLds fused_lds(int D, int H, int r, int q) {
    FusedLds L{};
    const int kgroups = fused_kgroups(D);
    const int hpad = (H + 4 * kFHid - 1) / (4 * kFHid) * (4 * kFHid);
    const int nft = (r + q + 31) / 32;
    L.xch = odd_at_least(8 * kgroups);
    L.tuch = odd_at_least(4 * nft);
    L.yp = D + 8;
    L.b1 = static_cast<size_t>(hpad) * 4;                    // a multiple of 1 KB
    L.b2 = (static_cast<size_t>(D) * 4 + 1023) / 1024 * 1024;
    // the x copy issues whole 64-lane rounds of slots: round its region up
    L.x = ((static_cast<size_t>(kFRows) * L.xch + 63) / 64) * 64 * 16;
    L.ring = static_cast<size_t>(4) * kNS * kStageBytes;
    // the four waves' partial sums of the larger reduction round
    // ((nft + 1) / 2 feature tiles, pitch 32 n + 4 floats per token)
    L.areas = static_cast<size_t>(4) * kFRows * (32 * ((nft + 1) / 2) + 4) * 4;
    L.yrows = static_cast<size_t>(kFRows) * L.yp * 2;
    L.epi_off = L.b1 + L.b2;                                 // past b2, which phase C reads
    L.tu_off = L.epi_off + ((L.areas > L.yrows ? L.areas : L.yrows) + 15) / 16 * 16;
    const size_t run = L.b1 + L.b2 + L.x + L.ring;
    const size_t tail = L.tu_off + static_cast<size_t>(kFRows) * L.tuch * 16;
    L.total = run > tail ? run : tail;
    return L;
}

}  // namespace

// Arrival counters of the hidden split start at zero in every launch (a fill
// kernel, so that the launch sequence records no memset).
__global__ void k_zero_counters(int32_t* c, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) c[i] = 0;
}

int fused_split(int64_t T, int E, int H) {
    const int64_t tiles = (T + kFRows - 1) / kFRows + E;
    const int64_t groups = (H + 4 * kFHid - 1) / (4 * kFHid);   // four-slice groups
    int64_t s = kFMaxSplit;
    if (256 / tiles < s) s = 256 / tiles;
    if (groups < s) s = groups;
    return s < 2 ? 1 : static_cast<int>(s);
}

size_t fused_part_bytes(int64_t T, int E, int H, int r, int q) {
    const int s = fused_split(T, E, H);
    if (s < 2) return 0;
    const int64_t tiles = (T + kFRows - 1) / kFRows + E;
    return static_cast<size_t>(tiles) * s * kFRows * (32 * ((r + q + 31) / 32)) * sizeof(float);
}

bool fused_top1_supported(int D, int H, int r, int q) {
    if (!(D >= 8 && D <= kFusedMaxD && H >= 8 && H <= kFusedMaxH && r % 32 == 0 && r + q > 0 &&
          r + q <= kFusedMaxRQ))
        return false;
    if (D > 128 * kCt) return false;               // one pass of y column tiles
    if (fused_kgroups(D) != kFGroups) return false;   // the compiled input-group count
    return fused_lds(D, H, r, q).total <= kLdsBytes - kStaticLds;
}

hipError_t launch_fused_top1(const void* x, const void* W1, const float* b1, const void* US,
                             const void* Vt, const float* b2, const void* P, const void* Q,
                             const int32_t* perm, const int32_t* offsets, const int32_t* idx,
                             const int32_t* tile_counts, const float* gate, void* y, int64_t T,
                             int D, int H, int E, int r, int q, float* part, int32_t* counters,
                             hipStream_t st, const ClassArgs* cls) {
    if (!fused_top1_supported(D, H, r, q)) return hipErrorInvalidValue;
    if (T == 0) return hipSuccess;
    const int split = fused_split(T, E, H);
    if (split > 1 && (part == nullptr || counters == nullptr)) return hipErrorInvalidValue;
    if (cls != nullptr && (split > 1 || !class_ffn_supported(cls->D, cls->H) || cls->D != D ||
                           cls->H != H || cls->nparts < 1))
        return hipErrorInvalidValue;
    FusedArgs a{};
    a.x = static_cast<const bf16_bits*>(x);
    a.W1 = static_cast<const bf16_bits*>(W1);
    a.b1 = b1;
    a.US = static_cast<const bf16_bits*>(US);
    a.Vt = static_cast<const bf16_bits*>(Vt);
    a.b2 = b2;
    a.P = static_cast<const bf16_bits*>(P);
    a.Q = static_cast<const bf16_bits*>(Q);
    a.perm = perm;
    a.offsets = offsets;
    a.idx = idx;
    a.tile_counts = tile_counts;
    a.htile = hist_tile(T, E);
    a.nh = static_cast<int>(hist_tiles(T, E));
    if (tile_counts != nullptr &&
        (idx == nullptr || static_cast<int64_t>(a.nh) * E > kInlineScanMax || E > 64))
        return hipErrorInvalidValue;
    a.gate = gate;
    a.y = static_cast<bf16_bits*>(y);
    a.T = T;
    a.D = D;
    a.H = H;
    a.E = E;
    a.r = r;
    a.q = q;
    a.hpad = (H + 4 * kFHid - 1) / (4 * kFHid) * (4 * kFHid);
    const int nft = (r + q + 31) / 32;
    const FusedLds L = fused_lds(D, H, r, q);
    a.xch = L.xch;
    a.tuch = L.tuch;
    a.yp = L.yp;
    a.b2_off = static_cast<int>(L.b1);
    a.b2_chunks = static_cast<int>(L.b2 / 16);
    a.x_off = static_cast<int>(L.b1 + L.b2);
    a.ring_off = static_cast<int>(L.b1 + L.b2 + L.x);
    a.epi_off = static_cast<int>(L.epi_off);
    a.tu_off = static_cast<int>(L.tu_off);
    const size_t lds = L.total;
    const int64_t tiles = (T + kFRows - 1) / kFRows + E;
    a.tiles_bound = static_cast<int>(tiles);
    a.split = split;
    a.part = part;
    a.counters = counters;
    // XCD-major workgroup order; a tile's S parts stay within one XCD (and
    // its L2), per_xcd being a multiple of S
    int per_xcd = static_cast<int>((tiles * split + kFXcds - 1) / kFXcds);
    per_xcd = (per_xcd + split - 1) / split * split;
    a.per_xcd = per_xcd;
    const int grid = a.per_xcd * kFXcds;
    if (split > 1) {
        // the fill kernel must not take the timing events meant for the
        // fused launch
        LaunchTiming& lt = launch_timing();
        const LaunchTiming keep = lt;
        lt = LaunchTiming{};
        launch_kernel(k_zero_counters, dim3((a.tiles_bound + 255) / 256), 256, 0, st, counters,
                      a.tiles_bound);
        lt = keep;
        const hipError_t err = hipGetLastError();
        if (err != hipSuccess) return err;
    }
    if (split > 1) return fused_launch_split(a, lds, grid, nft, st);
    if (cls != nullptr && cls->ncls > 0) {
        // the class rows' workgroups after the tiles' (their LDS plan is far
        // smaller than the tiles')
        const int64_t cgrid = grid + class_blocks(cls->ncls) * cls->nparts;
        if (cgrid > INT32_MAX || class_lds_bytes(H) > lds) return hipErrorInvalidValue;
        return fused_launch_cls(a, *cls, lds, static_cast<int>(cgrid), nft, st);
    }
    switch (nft) {
        case 1: return fused_cfg<1, false>(a, lds, grid, st);
        case 2: return fused_cfg<2, false>(a, lds, grid, st);
        case 3: return fused_cfg<3, false>(a, lds, grid, st);
        case 4: return fused_cfg<4, false>(a, lds, grid, st);
        default: return fused_cfg<5, false>(a, lds, grid, st);
    }
}

}  // namespace clearmoe
