// C ABI of the CLEAR-MoE FFN forward (declared in include/clearmoe.h).
// Host side only: argument checks (before any HIP call), workspace carving and
// the kernel sequence of each entry point on the caller's stream.
#include "clearmoe.h"

#include <stdint.h>

#include <mutex>
#include <vector>

#include "class_ffn.h"
#include "kernels.h"

using namespace clearmoe;

LaunchTiming& clearmoe::launch_timing() {
    thread_local LaunchTiming t;
    return t;
}

namespace {

constexpr size_t kAlign = 256;
constexpr int64_t kMaxDim = 1 << 16;

size_t up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Workspace layout.  Prefix shared by every entry point, then the buffers of
// the whole-layer forward.
struct Layout {
    size_t tile_counts, tile_base, chunk_tot;     // route / dispatch
    size_t counts, offsets, idx, gate, perm, inv;  // ffn_forward
    size_t z, tproj, hsh, u, hres, tu, fpart, fcount;
    size_t cpart, ccount;   // class rows' split over the hidden width: partial sums, arrivals
    // top-2 pair order (E * E <= kPairMaxKeys): keys, pair gates, the pair
    // permutation with its sort arrays, and [t|u_a|u_b] [T, r + 2q]
    size_t pkey, pgate, pperm, pinv, pcounts, poffsets, ptc, ptb, pct, ptu;
    size_t dispatch_end, total;
    // padded-batch backend only (after total): capacity E * T * k rows
    size_t perm_pad, inv_pad, seg, u_pad, hres_pad, padded_total;
};

size_t elem_size(int dtype) { return dtype == CLEARMOE_F32 ? 4 : 2; }

// Top-2 layers with few experts run in pair order: tokens sorted by their
// expert pair, one [t|u_a|u_b] product and one y product per pair segment.
bool pair_path(const clearmoe_shape& s) { return s.k == 2 && pair_keys(s.E) <= kPairMaxKeys; }

Layout layout(const clearmoe_shape& s) {
    Layout L{};
    const int64_t T = s.T, k = s.k, E = s.E;
    const int64_t ntiles = route_tiles(T);
    const int64_t nhist = E > 0 ? hist_tiles(T, static_cast<int>(E)) : 0;   // 64- or 256-token tiles
    const size_t es = elem_size(s.dtype);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off += up(bytes);
        return at;
    };
    // The histogram regions come first and depend on T and E only, so route and
    // dispatch calls with different D (or none) agree on where they are.
    L.tile_counts = take(sizeof(int32_t) * (nhist * E > 0 ? nhist * E : 1));
    L.tile_base = take(sizeof(int32_t) * (ntiles * E > 0 ? ntiles * E : 1));
    L.chunk_tot = take(sizeof(int32_t) * (scan_chunks(ntiles) * E > 0 ? scan_chunks(ntiles) * E : 1));
    L.dispatch_end = off;
    L.counts = take(sizeof(int32_t) * E);
    L.offsets = take(sizeof(int32_t) * (E + 1));
    L.idx = take(sizeof(int32_t) * T * k);
    L.gate = take(sizeof(float) * T * k);
    L.perm = take(sizeof(int32_t) * T * k);
    L.inv = take(sizeof(int32_t) * T * k);
    L.z = take(es * T * s.H);
    L.tproj = take(es * T * s.r);
    L.hsh = take(sizeof(float) * T * s.D);
    L.u = take(es * T * k * s.q);
    L.hres = take(sizeof(float) * T * k * s.D);
    L.tu = take(es * T * k * (s.r + s.q));
    if (pair_path(s)) {
        const int64_t P = pair_keys(static_cast<int>(E));
        L.pkey = take(sizeof(int32_t) * T);
        L.pgate = take(sizeof(float) * 2 * T);       // [2][T]: gates of a, of b
        L.pperm = take(sizeof(int32_t) * T);
        L.pinv = take(sizeof(int32_t) * T);
        L.pcounts = take(sizeof(int32_t) * P);
        L.poffsets = take(sizeof(int32_t) * (P + 1));
        L.ptc = take(sizeof(int32_t) * (T > 0 ? hist_tiles(T, static_cast<int>(P)) * P : 1));
        L.ptb = take(sizeof(int32_t) * (ntiles * P > 0 ? ntiles * P : 1));
        L.pct = take(sizeof(int32_t) * (scan_chunks(ntiles) * P > 0 ? scan_chunks(ntiles) * P : 1));
        L.ptu = take(es * T * (s.r + 2 * s.q));
    }
    // float32 partials and per-tile arrival counters: of the fused top-1
    // kernel's hidden split (small batches), or else, on the top-1 GEMM
    // chain, of the [t|u] product's split K
    // (a top-2 pair order's single-expert tokens take the top-1 path)
    const bool fused_ok = s.dtype == CLEARMOE_BF16 && fused_top1_supported(s.D, s.H, s.r, s.q);
    const bool top1 = k == 1 || pair_path(s);
    size_t fpart = 0, fcount = 0;
    if (top1 && fused_ok && T > 0) {
        fpart = fused_part_bytes(T, static_cast<int>(E), s.H, s.r, s.q);
        fcount = fpart > 0 ? static_cast<size_t>(T / 64 + E + 1) : 0;
    } else if (top1 && T > 0) {
        fpart = kGemmKsplitBytes;
        fcount = kGemmKsplitTiles;
    }
    L.fpart = take(fpart > 0 ? fpart : 1);
    L.fcount = take(sizeof(int32_t) * (fcount > 0 ? fcount : 1));
    L.cpart = take(kClsPartBytes);
    L.ccount = take(sizeof(uint64_t) * kClsCountWords);
    L.total = off;
    // A padded batch holds E sub-batches of the largest expert count, which
    // can be every assignment: room for E * T * k rows.
    const int64_t cap = E * T * k;
    L.perm_pad = take(sizeof(int32_t) * (cap > 0 ? cap : 1));
    L.inv_pad = take(sizeof(int32_t) * (T * k > 0 ? T * k : 1));
    L.seg = take(sizeof(int32_t) * (E + 1));
    L.u_pad = take(es * cap * s.q);
    L.hres_pad = take(sizeof(float) * cap * s.D);
    L.padded_total = off;
    return L;
}

// The regions clearmoe_ffn_forward (linear router, no class tokens) touches
// for this shape, packed: the fused top-1 path needs only the routing arrays
// (and, when it cannot dispatch in its own prologue, the dispatch arrays);
// the GEMM chains add their intermediates.  Regions a path does not touch
// keep offset 0 and are never read or written.
Layout layout_min(const clearmoe_shape& s) {
    Layout L{};
    const int64_t T = s.T, k = s.k, E = s.E;
    const size_t es = elem_size(s.dtype);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off += up(bytes > 0 ? bytes : 1);
        return at;
    };
    const bool fused = k == 1 && s.dtype == CLEARMOE_BF16 && fused_top1_supported(s.D, s.H, s.r, s.q);
    const bool own = fused && s.renorm && hist_tiles(T, static_cast<int>(E)) * E <= kInlineScanMax;
    const bool pair = pair_path(s);
    const int64_t ntiles = route_tiles(T);
    L.tile_counts = take(sizeof(int32_t) * hist_tiles(T, static_cast<int>(E)) * E);
    if (pair) {
        const int64_t P = pair_keys(static_cast<int>(E));
        L.idx = take(sizeof(int32_t) * T * k);
        L.gate = take(sizeof(float) * T * k);
        L.pkey = take(sizeof(int32_t) * T);
        L.pgate = take(sizeof(float) * 2 * T);       // [2][T]: gates of a, of b
        L.pperm = take(sizeof(int32_t) * T);
        L.pinv = take(sizeof(int32_t) * T);
        L.pcounts = take(sizeof(int32_t) * P);
        L.poffsets = take(sizeof(int32_t) * (P + 1));
        L.ptc = take(sizeof(int32_t) * hist_tiles(T, static_cast<int>(P)) * P);
        L.ptb = take(sizeof(int32_t) * ntiles * P);
        L.pct = take(sizeof(int32_t) * scan_chunks(ntiles) * P);
        L.z = take(es * T * s.H);
        L.ptu = take(es * T * (s.r + 2 * s.q));
        L.total = off;
        return L;
    }
    if (!own) {
        L.tile_base = take(sizeof(int32_t) * ntiles * E);
        L.chunk_tot = take(sizeof(int32_t) * scan_chunks(ntiles) * E);
        L.counts = take(sizeof(int32_t) * E);
        L.offsets = take(sizeof(int32_t) * (E + 1));
        L.perm = take(sizeof(int32_t) * T * k);
        L.inv = take(sizeof(int32_t) * T * k);
    }
    L.dispatch_end = off;
    L.idx = take(sizeof(int32_t) * T * k);
    L.gate = take(sizeof(float) * T * k);
    if (fused) {
        const size_t fpart = T > 0 ? fused_part_bytes(T, static_cast<int>(E), s.H, s.r, s.q) : 0;
        if (fpart > 0) {
            L.fpart = take(fpart);
            L.fcount = take(sizeof(int32_t) * static_cast<size_t>(T / 64 + E + 1));
        }
    } else if (k == 1) {
        L.z = take(es * T * s.H);
        L.tu = take(es * T * (s.r + s.q));
        L.fpart = take(kGemmKsplitBytes);
        L.fcount = take(sizeof(int32_t) * kGemmKsplitTiles);
    } else {
        L.z = take(es * T * s.H);
        L.tproj = take(es * T * s.r);
        L.hsh = take(sizeof(float) * T * s.D);
        L.u = take(es * T * k * s.q);
        L.hres = take(sizeof(float) * T * k * s.D);
    }
    L.total = off;
    return L;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Shape checks common to every entry point (which fields matter depends on
// the entry point; unused fields must still be in range).  D, H, r and q
// must be multiples of the elements of a 16-byte piece, except where the
// entry point takes other shapes (unaligned_ok): the layer entry points and
// routing pad them, dispatch and combine copy their rows element by element.
int check_shape(const clearmoe_shape* s, bool layer, bool unaligned_ok = false) {
    if (s == nullptr) return CLEARMOE_ERR_INVALID_ARG;
    if (s->dtype != CLEARMOE_F32 && s->dtype != CLEARMOE_BF16) return CLEARMOE_ERR_UNSUPPORTED;
    if (s->T < 0 || s->D < 1 || s->D > kMaxDim) return CLEARMOE_ERR_INVALID_ARG;
    if (s->E < 1 || s->E > 64 || s->k < 1 || s->k > s->E) return CLEARMOE_ERR_INVALID_ARG;
    if (s->renorm != 0 && s->renorm != 1) return CLEARMOE_ERR_INVALID_ARG;
    if (static_cast<int64_t>(s->T) * s->k >= (int64_t{1} << 31)) return CLEARMOE_ERR_INVALID_ARG;
    const int mult = unaligned_ok ? 1 : (s->dtype == CLEARMOE_F32 ? 4 : 8);
    if (s->D % mult != 0) return CLEARMOE_ERR_INVALID_ARG;
    if (layer) {
        if (s->H < 1 || s->H > kMaxDim || s->H % mult != 0) return CLEARMOE_ERR_INVALID_ARG;
        const int mn = s->D < s->H ? s->D : s->H;
        if (s->r < 0 || s->r > mn || s->q < 0 || s->q > mn) return CLEARMOE_ERR_INVALID_ARG;
        if (s->r % mult != 0 || s->q % mult != 0) return CLEARMOE_ERR_INVALID_ARG;
    }
    return CLEARMOE_OK;
}

// Unaligned layer shapes (D, H, r or q not a multiple of the elements of a
// 16-byte piece) run on zero-padded copies of their operands in the
// workspace.  Padding changes no result: an extra input feature or basis
// component multiplies zeros, and an extra hidden unit has z = GELU(0 + 0) =
// 0; the router's logits are the same sums, so the routing is the same, and
// the padded layer's y cropped to D columns is the layer's y.
int piece_elems(int dtype) { return dtype == CLEARMOE_F32 ? 4 : 8; }
int round_up(int v, int m) { return (v + m - 1) / m * m; }
bool unaligned_layer(const clearmoe_shape& s) {
    const int m = piece_elems(s.dtype);
    return s.D % m != 0 || s.H % m != 0 || s.r % m != 0 || s.q % m != 0;
}
clearmoe_shape aligned_shape(const clearmoe_shape& s) {
    const int m = piece_elems(s.dtype);
    clearmoe_shape a = s;
    a.D = round_up(s.D, m);
    a.H = round_up(s.H, m);
    a.r = round_up(s.r, m);
    a.q = round_up(s.q, m);
    return a;
}
// Workspace of an unaligned layer: the aligned layer's own workspace first,
// then the padded copies (every operand a layer entry point may take).
struct PadLayout {
    size_t inner, x, y, W1, b1, US, Vt, b2, P, Q, Wg, Wh, W2, total;
};
PadLayout pad_layout(const clearmoe_shape& s) {
    const clearmoe_shape a = aligned_shape(s);
    const size_t es = elem_size(s.dtype);
    const size_t T = static_cast<size_t>(s.T), E = static_cast<size_t>(s.E);
    const size_t D = static_cast<size_t>(a.D), H = static_cast<size_t>(a.H);
    const size_t r = static_cast<size_t>(a.r), q = static_cast<size_t>(a.q);
    PadLayout p{};
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        off = up(off + bytes);
        return o;
    };
    p.inner = take(layout(a).total);
    p.x = take(es * T * D);
    p.y = take(es * T * D);
    p.W1 = take(es * H * D);
    p.b1 = take(4 * H);
    p.US = take(es * D * r);
    p.Vt = take(es * r * H);
    p.b2 = take(4 * D);
    p.P = take(es * E * D * q);
    p.Q = take(es * E * q * H);
    p.Wg = take(es * E * D);
    p.Wh = take(es * static_cast<size_t>(kMlpHiddenMax) * D);
    p.W2 = take(es * D * H);
    p.total = off;
    return p;
}

// Routing with a row width D that is not a multiple of the elements of a
// 16-byte piece runs on padded copies of x and the router's input matrix
// (Wg, or an MLP router's Wh), placed after the aligned shape's own regions;
// a valid layer shape uses the layer's padded copies (pad_layout).
struct RoutePads {
    clearmoe_shape a;     // the aligned routing shape (H = r = q = 0)
    size_t x, Wg, Wh, total;
};
RoutePads route_pads(const clearmoe_shape& s) {
    RoutePads r{};
    r.a = s;
    r.a.D = round_up(s.D, piece_elems(s.dtype));
    r.a.H = r.a.r = r.a.q = 0;
    if (check_shape(&s, true, true) == CLEARMOE_OK) {
        const PadLayout p = pad_layout(s);
        r.x = p.x;
        r.Wg = p.Wg;
        r.Wh = p.Wh;
        r.total = p.total;
        return r;
    }
    const size_t es = elem_size(s.dtype), D = static_cast<size_t>(r.a.D);
    size_t off = up(layout(r.a).total);
    r.x = off;
    off = up(off + es * static_cast<size_t>(s.T) * D);
    r.Wg = off;
    off = up(off + es * static_cast<size_t>(s.E) * D);
    r.Wh = off;
    off = up(off + es * static_cast<size_t>(kMlpHiddenMax) * D);
    r.total = off;
    return r;
}
bool unaligned_rows(const clearmoe_shape& s) { return s.D % piece_elems(s.dtype) != 0; }
int route_unaligned(const clearmoe_shape& s, const clearmoe_router& router, const void* x,
                    int32_t* idx, float* gate, void* ws, size_t ws_bytes, hipStream_t st);

// ---- stage timing: two events per timed launch, recorded on its stream ----
struct StageTimer {
    bool on = false;
    unsigned mask = 0;
    int used = 0;
    int every = 1;     // time launches 0, every, 2 every, ... of the selected stages
    int64_t seen = 0;  // selected launches since timing started
    std::vector<hipEvent_t> ev;   // 2 per record
    std::vector<int> stage;
};
StageTimer g_timer;
std::mutex g_timer_mu;

class StageScope {
  public:
    StageScope(int stage, hipStream_t st) {
        (void)st;
        if (!g_timer.on || !((g_timer.mask >> stage) & 1u)) return;
        std::lock_guard<std::mutex> lk(g_timer_mu);
        if (g_timer.seen++ % g_timer.every != 0) return;
        if (g_timer.used >= static_cast<int>(g_timer.stage.size())) return;
        slot_ = g_timer.used++;
        g_timer.stage[slot_] = stage;
        launch_timing() = LaunchTiming{g_timer.ev[2 * slot_], g_timer.ev[2 * slot_ + 1]};
    }
    ~StageScope() {
        if (slot_ < 0) return;
        LaunchTiming& t = launch_timing();
        if (t.start == g_timer.ev[2 * slot_]) {   // no kernel took the events
            t = LaunchTiming{};
            std::lock_guard<std::mutex> lk(g_timer_mu);
            g_timer.stage[slot_] = -1;
        }
    }
    StageScope(const StageScope&) = delete;
    StageScope& operator=(const StageScope&) = delete;

  private:
    int slot_ = -1;
};

// Launch one stage under its timing scope.
#define CLEARMOE_STAGE(stage, st, expr)                  \
    do {                                                  \
        StageScope scope_(stage, st);                     \
        const hipError_t e_ = (expr);                     \
        if (e_ != hipSuccess) return CLEARMOE_ERR_HIP;    \
    } while (0)

template <typename P>
P* at(void* ws, size_t off) {
    return reinterpret_cast<P*>(static_cast<unsigned char*>(ws) + off);
}

clearmoe_router linear_router(const void* Wg, const float* bg) {
    clearmoe_router r{};
    r.Wg = Wg;
    r.bg = bg;
    return r;
}

// Router checks (before any HIP call).
// wa: the alignment the router's matrices need (16 bytes; one element when
// they are read into padded copies).
int check_router(const clearmoe_shape& s, const clearmoe_router* r, size_t wa = 16) {
    if (r == nullptr || r->Wg == nullptr || !aligned(r->Wg, wa)) return CLEARMOE_ERR_INVALID_ARG;
    if (r->bg && !aligned(r->bg, 4)) return CLEARMOE_ERR_INVALID_ARG;
    if (r->hidden < 0 || r->hidden > kMlpHiddenMax) return CLEARMOE_ERR_INVALID_ARG;
    if (r->hidden > 0 && (r->Wh == nullptr || !aligned(r->Wh, wa) || (r->bh && !aligned(r->bh, 4))))
        return CLEARMOE_ERR_INVALID_ARG;
    if (r->adaptive != 0 && r->adaptive != 1) return CLEARMOE_ERR_INVALID_ARG;
    if (r->adaptive && (s.k != 2 || s.E < 2 || r->tau != r->tau)) return CLEARMOE_ERR_INVALID_ARG;
    if (r->dense_stride < 0 || r->reserved != 0) return CLEARMOE_ERR_INVALID_ARG;
    if (r->W2 && !aligned(r->W2, wa)) return CLEARMOE_ERR_INVALID_ARG;
    return CLEARMOE_OK;
}

// Routing and the per-tile histogram (left in the workspace for dispatch).
int route_impl(const clearmoe_shape& s, const Layout& L, const clearmoe_router& rt, const void* x,
               int32_t* idx, float* gate, void* ws, hipStream_t st) {
    int32_t* tc = at<int32_t>(ws, L.tile_counts);
    if (rt.hidden == 0) {
        CLEARMOE_STAGE(CLEARMOE_STAGE_ROUTE, st,
                       launch_route(s.dtype, x, rt.Wg, rt.bg, s.T, s.D, s.E, s.k, rt.adaptive,
                                    s.renorm, rt.tau, rt.dense_stride, idx, gate, tc, st));
        return CLEARMOE_OK;
    }
    CLEARMOE_STAGE(CLEARMOE_STAGE_ROUTE, st,
                   launch_route_mlp(s.dtype, x, rt.Wh, rt.bh, rt.Wg, rt.bg, s.T, s.D, rt.hidden,
                                    s.E, s.k, rt.adaptive, s.renorm, rt.tau, rt.dense_stride,
                                    idx, gate, st));
    CLEARMOE_STAGE(CLEARMOE_STAGE_TILE_HIST, st,
                   launch_tile_histogram(idx, s.T, s.E, s.k, tc, st));
    return CLEARMOE_OK;
}

int dispatch_impl(const clearmoe_shape& s, const Layout& L, const int32_t* idx, void* ws,
                  int32_t* counts, int32_t* offsets, int32_t* perm, int32_t* inv, const void* x,
                  void* xperm, bool hist_in_ws, hipStream_t st) {
    if (x != nullptr && s.D % piece_elems(s.dtype) != 0) {
        // rows that are not whole 16-byte pieces: the indices first, then the
        // rows one element at a time
        const int rc = dispatch_impl(s, L, idx, ws, counts, offsets, perm, inv, nullptr, nullptr,
                                     hist_in_ws, st);
        if (rc != CLEARMOE_OK) return rc;
        CLEARMOE_STAGE(CLEARMOE_STAGE_PERMUTE, st,
                       launch_gather_rows_elem(s.dtype, x, perm, offsets + s.E,
                                               static_cast<int64_t>(s.T) * s.k, s.k, s.D, xperm, st));
        return CLEARMOE_OK;
    }
    int32_t* tc = at<int32_t>(ws, L.tile_counts);
    int32_t* tb = at<int32_t>(ws, L.tile_base);
    const int64_t nt = route_tiles(s.T);
    if (!hist_in_ws)
        CLEARMOE_STAGE(CLEARMOE_STAGE_TILE_HIST, st,
                       launch_tile_histogram(idx, s.T, s.E, s.k, tc, st));
    if (hist_tiles(s.T, s.E) * s.E <= kInlineScanMax) {
        // small histogram: the permutation scans it itself (one launch fewer)
        CLEARMOE_STAGE(CLEARMOE_STAGE_PERMUTE, st,
                       launch_permute(s.dtype, idx, tb, nullptr, offsets, tc, counts, s.T, s.E,
                                      s.k, perm, inv, x, xperm, s.D, st));
    } else {
        int32_t* ct = at<int32_t>(ws, L.chunk_tot);
        CLEARMOE_STAGE(CLEARMOE_STAGE_SCAN, st, launch_scan(tc, nt, s.E, tb, ct, st));
        CLEARMOE_STAGE(CLEARMOE_STAGE_PERMUTE, st,
                       launch_permute(s.dtype, idx, tb, ct, offsets, nullptr, counts, s.T, s.E,
                                      s.k, perm, inv, x, xperm, s.D, st));
    }
    return CLEARMOE_OK;
}

// Argument checks of the whole-layer entry points (before any HIP call).
int check_layer_args(const clearmoe_shape* shape, const void* x, const void* W1, const float* b1,
                     const void* US, const void* Vt, const float* b2, const void* P, const void* Q,
                     const void* Wg, const float* bg, const void* y, const int32_t* idx_out,
                     const float* gate_out) {
    int rc = check_shape(shape, true);
    if (rc != CLEARMOE_OK) return rc;
    const clearmoe_shape& s = *shape;
    if (!W1 || (s.T > 0 && (!x || !y))) return CLEARMOE_ERR_INVALID_ARG;
    if (s.r > 0 && (!US || !Vt)) return CLEARMOE_ERR_INVALID_ARG;
    if (s.q > 0 && (!P || !Q)) return CLEARMOE_ERR_INVALID_ARG;
    const void* v16[] = {x, W1, US, Vt, P, Q, Wg, y};
    for (const void* p : v16)
        if (p && !aligned(p, 16)) return CLEARMOE_ERR_INVALID_ARG;
    const void* v4[] = {b1, b2, bg, idx_out, gate_out};
    for (const void* p : v4)
        if (p && !aligned(p, 4)) return CLEARMOE_ERR_INVALID_ARG;
    return CLEARMOE_OK;
}

// z = GELU(x W1^T + b1), then the shared basis t = z Vt^T, h_sh = t US^T + b2
// (all in token order).
int shared_impl(const clearmoe_shape& s, const void* x, const void* W1, const float* b1,
                const void* US, const void* Vt, const float* b2, void* z, void* tproj, float* hsh,
                hipStream_t st) {
    GemmDesc g = gemm_desc(s.T, s.H, s.D);
    g.A = x; g.lda = s.D;
    g.B = W1; g.ldb = s.D;
    g.C = z; g.ldc = s.H; g.c_f32 = 0;
    g.bias = b1; g.gelu = 1;
    CLEARMOE_STAGE(CLEARMOE_STAGE_FC1, st, launch_gemm(s.dtype, g, st));
    g = gemm_desc(s.T, s.r, s.H);
    g.A = z; g.lda = s.H;
    g.B = Vt; g.ldb = s.H;
    g.C = tproj; g.ldc = s.r; g.c_f32 = 0;
    if (s.r > 0) CLEARMOE_STAGE(CLEARMOE_STAGE_BASIS_T, st, launch_gemm(s.dtype, g, st));
    g = gemm_desc(s.T, s.D, s.r);
    g.A = tproj; g.lda = s.r;
    g.B = US; g.ldb = s.r;
    g.C = hsh; g.ldc = s.D; g.c_f32 = 1;
    g.bias = b2;
    CLEARMOE_STAGE(CLEARMOE_STAGE_BASIS_H, st, launch_gemm(s.dtype, g, st));
    return CLEARMOE_OK;
}

// Residual over row segments seg[0..E] of a row order given by rows (-1 =
// padding row, which reads zeros):  u = gate * (z[rows/k] Q_e^T) ;
// h_res = u P_e^T  (M rows in all).
int residual_impl(const clearmoe_shape& s, int64_t M, const void* z, const int32_t* rows,
                  const int32_t* seg, const float* gate, const void* P, const void* Q, void* u,
                  float* hres, hipStream_t st) {
    GemmDesc g = gemm_desc(M, s.q, s.H);
    g.A = z; g.lda = s.H; g.a_rows = rows; g.a_div = s.k;
    g.B = Q; g.ldb = s.H; g.b_seg_stride = static_cast<int64_t>(s.q) * s.H;
    g.C = u; g.ldc = s.q; g.c_f32 = 0;
    g.row_scale = gate; g.scale_rows = rows;
    g.seg_offsets = seg; g.nseg = s.E;
    if (s.q > 0) CLEARMOE_STAGE(CLEARMOE_STAGE_RES_U, st, launch_gemm(s.dtype, g, st));
    g = gemm_desc(M, s.D, s.q);
    g.A = u; g.lda = s.q;
    g.B = P; g.ldb = s.q; g.b_seg_stride = static_cast<int64_t>(s.D) * s.q;
    g.C = hres; g.ldc = s.D; g.c_f32 = 1;
    g.seg_offsets = seg; g.nseg = s.E;
    CLEARMOE_STAGE(CLEARMOE_STAGE_RES_H, st, launch_gemm(s.dtype, g, st));
    return CLEARMOE_OK;
}

// Pinned host copy of the expert counts (padded backend), one per thread.
thread_local int32_t* t_host_counts = nullptr;

// A side stream per device (default priority, created on first use and kept
// until the process ends) on which work that does not depend on the routing
// runs beside it: fork = an event recorded on the caller's stream that the
// side stream waits for; join = an event recorded on the side stream that
// the caller's stream waits for, so the call's work stays ordered on the
// caller's stream as a whole.  One call forks and joins under g_side_mu.
struct SideStream {
    hipStream_t s = nullptr;
    hipEvent_t fork = nullptr, join = nullptr;
};
std::mutex g_side_mu;
std::vector<SideStream> g_side;

int side_stream(SideStream** out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return CLEARMOE_ERR_HIP;
    if (static_cast<size_t>(dev) >= g_side.size()) g_side.resize(static_cast<size_t>(dev) + 1);
    SideStream& ss = g_side[static_cast<size_t>(dev)];
    if (ss.s == nullptr) {
        if (hipStreamCreateWithFlags(&ss.s, hipStreamNonBlocking) != hipSuccess) {
            ss.s = nullptr;
            return CLEARMOE_ERR_HIP;
        }
        if (hipEventCreateWithFlags(&ss.fork, hipEventDisableTiming) != hipSuccess ||
            hipEventCreateWithFlags(&ss.join, hipEventDisableTiming) != hipSuccess)
            return CLEARMOE_ERR_HIP;
    }
    *out = &ss;
    return CLEARMOE_OK;
}

}  // namespace

#ifndef CLEARMOE_SOURCE_DIGEST
#define CLEARMOE_SOURCE_DIGEST "0000000000000000"
#endif
// The digest of the sources this library was built from, after a marker that
// the build scripts find in the file without loading it.
__attribute__((used)) const char g_source_digest[] = "CLEARMOE-SOURCE-DIGEST=" CLEARMOE_SOURCE_DIGEST;

extern "C" {

int clearmoe_version(void) { return (0 << 16) | 3; }

const char* clearmoe_source_digest(void) {
    return g_source_digest + sizeof("CLEARMOE-SOURCE-DIGEST=") - 1;
}

const char* clearmoe_status_string(int status) {
    switch (status) {
        case CLEARMOE_OK: return "ok";
        case CLEARMOE_ERR_INVALID_ARG: return "invalid argument";
        case CLEARMOE_ERR_UNSUPPORTED: return "unsupported";
        case CLEARMOE_ERR_WORKSPACE: return "workspace missing or too small";
        case CLEARMOE_ERR_HIP: return "HIP launch failed";
        case CLEARMOE_ERR_TOO_LARGE:
            return "shape needs more scratch than the no-allocation entry point holds";
        default: return "unknown status";
    }
}

size_t clearmoe_workspace_bytes(const clearmoe_shape* shape) {
    if (shape != nullptr && check_shape(shape, true, true) == CLEARMOE_OK && unaligned_layer(*shape))
        return pad_layout(*shape).total;
    if (shape != nullptr && check_shape(shape, false, true) == CLEARMOE_OK && unaligned_rows(*shape))
        return route_pads(*shape).total;     // route / dispatch-only shape
    if (check_shape(shape, false) != CLEARMOE_OK) return 0;
    clearmoe_shape s = *shape;
    if (check_shape(shape, true) != CLEARMOE_OK) {  // route / dispatch-only shape
        s.H = 0;
        s.r = 0;
        s.q = 0;
    }
    return layout(s).total;
}

int clearmoe_route(const clearmoe_shape* shape, const void* x, const void* Wg, const float* bg,
                   int32_t* idx, float* gate, void* ws, size_t ws_bytes, hipStream_t stream) {
    int rc = check_shape(shape, false, true);
    if (rc != CLEARMOE_OK) return rc;
    const clearmoe_shape& s = *shape;
    if (unaligned_rows(s))
        return route_unaligned(s, linear_router(Wg, bg), x, idx, gate, ws, ws_bytes, stream);
    const bool tok = s.T > 0;                 // per-token arrays may be NULL when T == 0
    if (!Wg || (tok && (!x || !idx || !gate))) return CLEARMOE_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(Wg, 16) || !aligned(idx, 4) || !aligned(gate, 4) ||
        (bg && !aligned(bg, 4)))
        return CLEARMOE_ERR_INVALID_ARG;
    clearmoe_shape sl = s;
    sl.H = sl.r = sl.q = 0;
    const Layout L = layout(sl);
    if (!ws || !aligned(ws, kAlign) || ws_bytes < L.dispatch_end) return CLEARMOE_ERR_WORKSPACE;
    return route_impl(s, L, linear_router(Wg, bg), x, idx, gate, ws, stream);
}

int clearmoe_route_ex(const clearmoe_shape* shape, const clearmoe_router* router, const void* x,
                      int32_t* idx, float* gate, void* ws, size_t ws_bytes, hipStream_t stream) {
    int rc = check_shape(shape, false, true);
    if (rc != CLEARMOE_OK) return rc;
    const clearmoe_shape& s = *shape;
    if (unaligned_rows(s)) {
        rc = check_router(s, router, elem_size(s.dtype));
        if (rc != CLEARMOE_OK) return rc;
        return route_unaligned(s, *router, x, idx, gate, ws, ws_bytes, stream);
    }
    rc = check_router(s, router);
    if (rc != CLEARMOE_OK) return rc;
    const bool tok = s.T > 0;
    if (tok && (!x || !idx || !gate)) return CLEARMOE_ERR_INVALID_ARG;
    if (!aligned(x, 16) || !aligned(idx, 4) || !aligned(gate, 4)) return CLEARMOE_ERR_INVALID_ARG;
    clearmoe_shape sl = s;
    sl.H = sl.r = sl.q = 0;
    const Layout L = layout(sl);
    if (!ws || !aligned(ws, kAlign) || ws_bytes < L.dispatch_end) return CLEARMOE_ERR_WORKSPACE;
    return route_impl(s, L, *router, x, idx, gate, ws, stream);
}

int clearmoe_dispatch(const clearmoe_shape* shape, const int32_t* idx, void* ws, size_t ws_bytes,
                      int32_t* counts, int32_t* offsets, int32_t* perm, int32_t* inv,
                      const void* x, void* xperm, unsigned flags, hipStream_t stream) {
    int rc = check_shape(shape, false, true);
    if (rc != CLEARMOE_OK) return rc;
    const clearmoe_shape& s = *shape;
    const bool tok = s.T > 0;
    if (!counts || !offsets || (tok && (!idx || !perm || !inv))) return CLEARMOE_ERR_INVALID_ARG;
    if (tok && (x == nullptr) != (xperm == nullptr)) return CLEARMOE_ERR_INVALID_ARG;
    // rows that are whole 16-byte pieces are copied as such; others element
    // by element
    const size_t ra = unaligned_rows(s) ? elem_size(s.dtype) : 16;
    if (!aligned(idx, 4) || !aligned(counts, 4) || !aligned(offsets, 4) || !aligned(perm, 4) ||
        !aligned(inv, 4) || (x && (!aligned(x, ra) || !aligned(xperm, ra))))
        return CLEARMOE_ERR_INVALID_ARG;
    if (flags & ~static_cast<unsigned>(CLEARMOE_DISPATCH_HIST_IN_WS)) return CLEARMOE_ERR_INVALID_ARG;
    clearmoe_shape sl = s;
    sl.D = round_up(s.D, piece_elems(s.dtype));
    sl.H = sl.r = sl.q = 0;
    const Layout L = layout(sl);
    if (!ws || !aligned(ws, kAlign) || ws_bytes < L.dispatch_end) return CLEARMOE_ERR_WORKSPACE;
    return dispatch_impl(s, L, idx, ws, counts, offsets, perm, inv, x, xperm,
                         (flags & CLEARMOE_DISPATCH_HIST_IN_WS) != 0, stream);
}

int clearmoe_combine(const clearmoe_shape* shape, const void* ye, const int32_t* inv,
                     const float* gate, void* y, hipStream_t stream) {
    int rc = check_shape(shape, false, true);
    if (rc != CLEARMOE_OK) return rc;
    const clearmoe_shape& s = *shape;
    if (s.T > 0 && (!ye || !inv || !gate || !y)) return CLEARMOE_ERR_INVALID_ARG;
    const size_t ra = unaligned_rows(s) ? elem_size(s.dtype) : 16;
    if (!aligned(ye, ra) || !aligned(y, ra) || !aligned(inv, 4) || !aligned(gate, 4))
        return CLEARMOE_ERR_INVALID_ARG;
    if (unaligned_rows(s)) {
        CLEARMOE_STAGE(CLEARMOE_STAGE_COMBINE, stream,
                       launch_combine_gated_elem(s.dtype, ye, inv, gate, y, s.T, s.D, s.k, stream));
        return CLEARMOE_OK;
    }
    CLEARMOE_STAGE(CLEARMOE_STAGE_COMBINE, stream,
                   launch_combine_gated(s.dtype, ye, inv, gate, y, s.T, s.D, s.k, stream));
    return CLEARMOE_OK;
}

}  // extern "C"

namespace {

// Class tokens (every dense_stride-th token, from token 0) on the dense path:
// y[c] = GELU(x[c] W1^T + b1) W2^T + b2 over the ceil(T / dense_stride) class
// rows, which the strided leading dimensions pick out of x and y.  With
// z_all the token-order z of the whole layer is already there (its class
// rows are read with a stride); otherwise fc1 + GELU runs on the class rows
// into the workspace's z region first.
int class_tokens_impl(const clearmoe_shape& s, const clearmoe_router& rt, const void* x,
                      const void* W1, const float* b1, const float* b2, void* z, bool z_all,
                      void* y, const Layout& L, void* ws, hipStream_t st) {
    const int64_t sd = rt.dense_stride;
    const int64_t ncls = (s.T + sd - 1) / sd;
    int64_t zld = s.H;
    if (!z_all && s.dtype == CLEARMOE_BF16 && class_ffn_supported(s.D, s.H)) {
        // both products in one pass per 32 class rows (z stays on chip)
        ClassArgs c{};
        c.x = static_cast<const bf16_bits*>(x);
        c.W1 = static_cast<const bf16_bits*>(W1);
        c.b1 = b1;
        c.W2 = static_cast<const bf16_bits*>(rt.W2);
        c.b2 = b2;
        c.y = static_cast<bf16_bits*>(y);
        c.ncls = ncls;
        c.stride = sd;
        c.D = s.D;
        c.H = s.H;
        class_ffn_plan(c, at<float>(ws, L.cpart), at<uint64_t>(ws, L.ccount));
        CLEARMOE_STAGE(CLEARMOE_STAGE_DENSE_FC2, st, launch_class_ffn(c, st));
        return CLEARMOE_OK;
    }
    if (z_all) {
        zld = static_cast<int64_t>(s.H) * sd;
    } else {
        GemmDesc g = gemm_desc(ncls, s.H, s.D);
        g.A = x; g.lda = static_cast<int64_t>(s.D) * sd;
        g.B = W1; g.ldb = s.D;
        g.C = z; g.ldc = s.H; g.c_f32 = 0;
        g.bias = b1; g.gelu = 1;
        CLEARMOE_STAGE(CLEARMOE_STAGE_FC1, st, launch_gemm(s.dtype, g, st));
    }
    GemmDesc g = gemm_desc(ncls, s.D, s.H);
    g.A = z; g.lda = zld;
    g.B = rt.W2; g.ldb = s.H;
    g.C = y; g.ldc = static_cast<int64_t>(s.D) * sd; g.c_f32 = 0;
    g.bias = b2;
    CLEARMOE_STAGE(CLEARMOE_STAGE_DENSE_FC2, st, launch_gemm(s.dtype, g, st));
    return CLEARMOE_OK;
}

int ffn_forward_impl(const clearmoe_shape* shape, const clearmoe_router* router, const void* x,
                     const void* W1, const float* b1, const void* US, const void* Vt,
                     const float* b2, const void* P, const void* Q, void* y, int32_t* idx_out,
                     float* gate_out, void* ws, size_t ws_bytes, hipStream_t stream,
                     const Layout* packed = nullptr) {
    int rc = check_layer_args(shape, x, W1, b1, US, Vt, b2, P, Q, nullptr, nullptr, y, idx_out,
                              gate_out);
    if (rc != CLEARMOE_OK) return rc;
    const clearmoe_shape& s = *shape;
    rc = check_router(s, router);
    if (rc != CLEARMOE_OK) return rc;
    if (router->dense_stride > 0 && router->W2 == nullptr) return CLEARMOE_ERR_INVALID_ARG;
    // a packed layout (no-allocation variant) serves only the linear router
    // without class tokens, whose regions it holds
    if (packed != nullptr && (router->hidden != 0 || router->adaptive || router->dense_stride > 0))
        return CLEARMOE_ERR_INVALID_ARG;
    const Layout L = packed != nullptr ? *packed : layout(s);
    if (!ws || !aligned(ws, kAlign) || ws_bytes < L.total) return CLEARMOE_ERR_WORKSPACE;
    if (s.T == 0) return CLEARMOE_OK;

    hipStream_t st = stream;
    const int64_t T = s.T, A = T * s.k;
    const bool cls = router->dense_stride > 0;
    const bool fused = s.k == 1 && s.dtype == CLEARMOE_BF16 && fused_top1_supported(s.D, s.H, s.r, s.q);
    int32_t* idx = idx_out ? idx_out : at<int32_t>(ws, L.idx);
    float* gate = gate_out ? gate_out : at<float>(ws, L.gate);
    int32_t* counts = at<int32_t>(ws, L.counts);
    int32_t* offsets = at<int32_t>(ws, L.offsets);
    int32_t* perm = at<int32_t>(ws, L.perm);
    int32_t* inv = at<int32_t>(ws, L.inv);
    void* z = at<void>(ws, L.z);
    void* tproj = at<void>(ws, L.tproj);
    float* hsh = at<float>(ws, L.hsh);
    void* u = at<void>(ws, L.u);
    float* hres = at<float>(ws, L.hres);

    // With the fused top-1 kernel the class tokens' dense path needs only x.
    // Without the hidden split it runs inside the fused launch; with it (a
    // small batch), on a side stream beside routing, dispatch and the fused
    // kernel (which leave compute units idle), into the workspace's z region
    // (unused by the fused path).
    std::unique_lock<std::mutex> side_lock;
    SideStream* side = nullptr;
    // whatever happens below, the caller's stream waits for the side work
    struct JoinGuard {
        hipStream_t st;
        SideStream** side;
        bool done = false;
        ~JoinGuard() {
            if (!done && *side != nullptr) (void)hipStreamWaitEvent(st, (*side)->join, 0);
        }
    } join_guard{st, &side};
    // The fused launch without the hidden split runs the class rows itself,
    // on workgroups past its tiles.
    const bool cls_in_fused = cls && fused && s.dtype == CLEARMOE_BF16 && fused_split(T, s.E, s.H) == 1 &&
                              class_ffn_supported(s.D, s.H);
    if (cls && fused && !cls_in_fused) {
        side_lock = std::unique_lock<std::mutex>(g_side_mu);
        rc = side_stream(&side);
        if (rc != CLEARMOE_OK) return rc;
        if (hipEventRecord(side->fork, st) != hipSuccess ||
            hipStreamWaitEvent(side->s, side->fork, 0) != hipSuccess)
            return CLEARMOE_ERR_HIP;
        rc = class_tokens_impl(s, *router, x, W1, b1, b2, z, false, y, L, ws, side->s);
        if (rc != CLEARMOE_OK) return rc;
        if (hipEventRecord(side->join, side->s) != hipSuccess) return CLEARMOE_ERR_HIP;
    }
    // Top-2 in pair order with every token on two experts: fc1 + GELU in
    // token order needs only x, so it runs on the side stream while routing
    // and the pair dispatch run here (they leave most of the chip idle); the
    // pair products wait for it.
    // (not in the no-allocation variant: it creates no stream or event)
    const bool fc1_aside = pair_path(s) && !router->adaptive && T > 0 && packed == nullptr;
    if (fc1_aside) {
        side_lock = std::unique_lock<std::mutex>(g_side_mu);
        rc = side_stream(&side);
        if (rc != CLEARMOE_OK) return rc;
        if (hipEventRecord(side->fork, st) != hipSuccess ||
            hipStreamWaitEvent(side->s, side->fork, 0) != hipSuccess)
            return CLEARMOE_ERR_HIP;
        GemmDesc g = gemm_desc(T, s.H, s.D);
        g.A = x; g.lda = s.D;
        g.B = W1; g.ldb = s.D;
        g.C = z; g.ldc = s.H; g.c_f32 = 0;
        g.bias = b1; g.gelu = 1;
        CLEARMOE_STAGE(CLEARMOE_STAGE_FC1, side->s, launch_gemm(s.dtype, g, side->s));
        if (hipEventRecord(side->join, side->s) != hipSuccess) return CLEARMOE_ERR_HIP;
    }

    // 1. router + top-k + per-tile histogram; 2. scan + stable permutation
    // (the fused top-1 kernel does the latter itself from the histogram
    // when it is small enough for one workgroup's scan; the pair order
    // dispatches pair keys instead, below)
    rc = route_impl(s, L, *router, x, idx, gate, ws, st);
    if (rc != CLEARMOE_OK) return rc;
    // (the fused kernel's own dispatch takes every top-1 gate as 1, which
    // holds for renormalised gates only; with renorm == 0 it reads them
    // from the dispatch kernels' order)
    const bool own_dispatch = fused && s.renorm && hist_tiles(T, s.E) * s.E <= kInlineScanMax;
    if (!own_dispatch && !pair_path(s)) {
        rc = dispatch_impl(s, L, idx, ws, counts, offsets, perm, inv, nullptr, nullptr, true, st);
        if (rc != CLEARMOE_OK) return rc;
    }

    // Top-1 in bf16: fc1 + GELU, [t|u] and y in one kernel (z stays on chip).
    if (fused) {
        const int32_t* tc = own_dispatch ? at<int32_t>(ws, L.tile_counts) : nullptr;
        ClassArgs c{};
        if (cls_in_fused) {
            c.x = static_cast<const bf16_bits*>(x);
            c.W1 = static_cast<const bf16_bits*>(W1);
            c.b1 = b1;
            c.W2 = static_cast<const bf16_bits*>(router->W2);
            c.b2 = b2;
            c.y = static_cast<bf16_bits*>(y);
            c.ncls = (T + router->dense_stride - 1) / router->dense_stride;
            c.stride = router->dense_stride;
            c.D = s.D;
            c.H = s.H;
            class_ffn_plan(c, at<float>(ws, L.cpart), at<uint64_t>(ws, L.ccount));
        }
        CLEARMOE_STAGE(CLEARMOE_STAGE_FUSED_TOP1, st,
                       launch_fused_top1(x, W1, b1, US, Vt, b2, P, Q, perm, offsets,
                                         own_dispatch ? idx : nullptr, tc, gate, y, T, s.D, s.H,
                                         s.E, s.r, s.q, at<float>(ws, L.fpart),
                                         at<int32_t>(ws, L.fcount), st, cls_in_fused ? &c : nullptr));
        // join: the class rows of y (written on the side stream) are complete
        // before anything later on the caller's stream
        if (side != nullptr) {
            join_guard.done = true;
            if (hipStreamWaitEvent(st, side->join, 0) != hipSuccess) return CLEARMOE_ERR_HIP;
        }
        return CLEARMOE_OK;
    }

    if (s.k == 1) {
        // 3. z = GELU(x W1^T + b1), token order
        GemmDesc g = gemm_desc(T, s.H, s.D);
        g.A = x; g.lda = s.D;
        g.B = W1; g.ldb = s.D;
        g.C = z; g.ldc = s.H; g.c_f32 = 0;
        g.bias = b1; g.gelu = 1;
        CLEARMOE_STAGE(CLEARMOE_STAGE_FC1, st, launch_gemm(s.dtype, g, st));

        // Top-1: every row p of the expert order is one token, so the shared
        // basis and the residual merge into two grouped products over p:
        //   [t | u](p) = z[perm p] [Vt ; Q_e]^T, the u columns scaled by the gate;
        //   y[perm p]  = [t | u](p) [US | P_e]^T + b2   (each y row written once).
        void* tu = at<void>(ws, L.tu);
        const int rq = s.r + s.q;
        g = gemm_desc(A, rq, s.H);
        g.A = z; g.lda = s.H; g.a_rows = perm; g.a_div = 1;
        g.B = Vt; g.ldb = s.H; g.b_seg_stride = 0;
        g.B1 = Q; g.ldb1 = s.H; g.b1_seg_stride = static_cast<int64_t>(s.q) * s.H;
        g.n_split = s.r;
        g.C = tu; g.ldc = rq; g.c_f32 = 0;
        g.row_scale = gate; g.scale_rows = perm; g.scale_col0 = s.r;
        g.seg_offsets = offsets; g.nseg = s.E;
        g.ks_part = at<float>(ws, L.fpart); g.ks_count = at<int32_t>(ws, L.fcount);
        if (rq > 0) CLEARMOE_STAGE(CLEARMOE_STAGE_TU, st, launch_gemm(s.dtype, g, st));
        g = gemm_desc(A, s.D, rq);
        g.A = tu; g.lda = rq;
        g.B = US; g.ldb = s.r; g.b_seg_stride = 0;
        g.B1 = P; g.ldb1 = s.q; g.b1_seg_stride = static_cast<int64_t>(s.D) * s.q;
        g.k_split = s.r;
        g.C = y; g.ldc = s.D; g.c_f32 = 0;
        g.c_rows = perm; g.c_div = 1;
        g.bias = b2;
        g.seg_offsets = offsets; g.nseg = s.E;
        CLEARMOE_STAGE(CLEARMOE_STAGE_Y, st, launch_gemm(s.dtype, g, st));
        if (cls) return class_tokens_impl(s, *router, x, W1, b1, b2, z, true, y, L, ws, st);
        return CLEARMOE_OK;
    }

    if (pair_path(s)) {
        // Top-2 in pair order.  Tokens are sorted by key: first the tokens
        // with one expert e (key e; only an adaptive router leaves a slot
        // empty), then those with two experts {a, b}, a < b (key E + the
        // pair's number).  Each pair segment merges the shared basis and both
        // residuals into two grouped products over the pair order p:
        //   [t | u_a | u_b](p) = z[pt] [Vt ; Q_a ; Q_b]^T, u_a times gate_a,
        //                        u_b times gate_b;
        //   y[pt] = [t | u_a | u_b](p) [US | P_a | P_b]^T + b2,
        // with pt = pperm[p]: each y row is written once, and neither h_sh
        // nor h_res is formed.  Single-expert tokens take the top-1 path over
        // the first E segments (the fused kernel where it applies).
        const int nkeys = pair_keys(s.E), npairs = nkeys - s.E;
        int32_t* pkey = at<int32_t>(ws, L.pkey);
        float* pga = at<float>(ws, L.pgate);
        float* pgb = pga + T;
        int32_t* pperm = at<int32_t>(ws, L.pperm);
        int32_t* poffsets = at<int32_t>(ws, L.poffsets);
        CLEARMOE_STAGE(CLEARMOE_STAGE_PAIR_KEY, st,
                       launch_pair_key(idx, gate, T, s.E, pkey, pga, pgb, at<int32_t>(ws, L.ptc), st));
        clearmoe_shape sp = s;
        sp.E = nkeys;
        sp.k = 1;
        Layout Lp = L;
        Lp.tile_counts = L.ptc;
        Lp.tile_base = L.ptb;
        Lp.chunk_tot = L.pct;
        rc = dispatch_impl(sp, Lp, pkey, ws, at<int32_t>(ws, L.pcounts), poffsets, pperm,
                           at<int32_t>(ws, L.pinv), nullptr, nullptr, true, st);
        if (rc != CLEARMOE_OK) return rc;
        const bool singles = router->adaptive != 0;
        const bool fused_ok = s.dtype == CLEARMOE_BF16 && fused_top1_supported(s.D, s.H, s.r, s.q);
        const int32_t* pair_seg = poffsets + s.E;
        GemmDesc g;
        bool z_pair_order = false;
        if (singles && fused_ok) {
            // single-expert tokens: the fused top-1 kernel over the first E
            // segments, with the gate of their one expert
            CLEARMOE_STAGE(CLEARMOE_STAGE_FUSED_TOP1, st,
                           launch_fused_top1(x, W1, b1, US, Vt, b2, P, Q, pperm, poffsets, nullptr,
                                             nullptr, pga, y, T, s.D, s.H, s.E, s.r, s.q,
                                             at<float>(ws, L.fpart), at<int32_t>(ws, L.fcount), st));
            // two-expert tokens: fc1 + GELU on their rows only, z in pair order
            g = gemm_desc(T, s.H, s.D);
            g.A = x; g.lda = s.D; g.a_rows = pperm; g.a_div = 1;
            g.B = W1; g.ldb = s.D;
            g.C = z; g.ldc = s.H; g.c_f32 = 0;
            g.bias = b1; g.gelu = 1;
            g.seg_offsets = pair_seg; g.nseg = npairs; g.seg_merge = 1;
            CLEARMOE_STAGE(CLEARMOE_STAGE_FC1, st, launch_gemm(s.dtype, g, st));
            z_pair_order = true;
        } else {
            if (!fc1_aside) {
                g = gemm_desc(T, s.H, s.D);
                g.A = x; g.lda = s.D;
                g.B = W1; g.ldb = s.D;
                g.C = z; g.ldc = s.H; g.c_f32 = 0;
                g.bias = b1; g.gelu = 1;
                CLEARMOE_STAGE(CLEARMOE_STAGE_FC1, st, launch_gemm(s.dtype, g, st));
            }
            if (singles) {
                // single-expert tokens: the top-1 chain's two grouped products
                void* tu = at<void>(ws, L.tu);
                const int rq = s.r + s.q;
                g = gemm_desc(T, rq, s.H);
                g.A = z; g.lda = s.H; g.a_rows = pperm; g.a_div = 1;
                g.B = Vt; g.ldb = s.H;
                g.B1 = Q; g.ldb1 = s.H; g.b1_seg_stride = static_cast<int64_t>(s.q) * s.H;
                g.n_split = s.r;
                g.C = tu; g.ldc = rq; g.c_f32 = 0;
                g.row_scale = pga; g.scale_rows = pperm; g.scale_col0 = s.r;
                g.seg_offsets = poffsets; g.nseg = s.E;
                g.ks_part = at<float>(ws, L.fpart); g.ks_count = at<int32_t>(ws, L.fcount);
                if (rq > 0) CLEARMOE_STAGE(CLEARMOE_STAGE_TU, st, launch_gemm(s.dtype, g, st));
                g = gemm_desc(T, s.D, rq);
                g.A = tu; g.lda = rq;
                g.B = US; g.ldb = s.r;
                g.B1 = P; g.ldb1 = s.q; g.b1_seg_stride = static_cast<int64_t>(s.D) * s.q;
                g.k_split = s.r;
                g.C = y; g.ldc = s.D; g.c_f32 = 0;
                g.c_rows = pperm; g.c_div = 1;
                g.bias = b2;
                g.seg_offsets = poffsets; g.nseg = s.E;
                CLEARMOE_STAGE(CLEARMOE_STAGE_Y, st, launch_gemm(s.dtype, g, st));
            }
        }
        if (fc1_aside) {   // z from the side stream
            join_guard.done = true;
            if (hipStreamWaitEvent(st, side->join, 0) != hipSuccess) return CLEARMOE_ERR_HIP;
        }
        void* ptu = at<void>(ws, L.ptu);
        const int rqq = s.r + 2 * s.q;
        g = gemm_desc(T, rqq, s.H);
        g.A = z; g.lda = s.H;
        if (!z_pair_order) {
            g.a_rows = pperm; g.a_div = 1;
        }
        g.B = Vt; g.ldb = s.H;
        g.B1 = Q; g.ldb1 = s.H; g.b1_seg_stride = static_cast<int64_t>(s.q) * s.H;
        g.B2 = Q; g.ldb2 = s.H; g.b2_seg_stride = static_cast<int64_t>(s.q) * s.H;
        g.n_split = s.r; g.n_split2 = s.r + s.q; g.pair_E = s.E;
        g.C = ptu; g.ldc = rqq; g.c_f32 = 0;
        g.row_scale = pga; g.row_scale2 = pgb; g.scale_rows = pperm;
        g.scale_col0 = s.r; g.scale_col1 = s.r + s.q;
        g.seg_offsets = pair_seg; g.nseg = npairs;
        if (rqq > 0) CLEARMOE_STAGE(CLEARMOE_STAGE_TU_PAIR, st, launch_gemm(s.dtype, g, st));
        g = gemm_desc(T, s.D, rqq);
        g.A = ptu; g.lda = rqq;
        g.B = US; g.ldb = s.r;
        g.B1 = P; g.ldb1 = s.q; g.b1_seg_stride = static_cast<int64_t>(s.D) * s.q;
        g.B2 = P; g.ldb2 = s.q; g.b2_seg_stride = static_cast<int64_t>(s.D) * s.q;
        g.k_split = s.r; g.k_split2 = s.r + s.q; g.pair_E = s.E;
        g.C = y; g.ldc = s.D; g.c_f32 = 0;
        g.c_rows = pperm; g.c_div = 1;
        g.bias = b2;
        g.seg_offsets = pair_seg; g.nseg = npairs;
        CLEARMOE_STAGE(CLEARMOE_STAGE_Y_PAIR, st, launch_gemm(s.dtype, g, st));
        // class tokens: their dense FFN output, from the token-order z when
        // there is one
        if (cls) return class_tokens_impl(s, *router, x, W1, b1, b2, z, !z_pair_order, y, L, ws, st);
        return CLEARMOE_OK;
    }

    // 3. z = GELU(x W1^T + b1); 4. shared basis t = z Vt^T, h_sh = t US^T + b2
    rc = shared_impl(s, x, W1, b1, US, Vt, b2, z, tproj, hsh, st);
    if (rc != CLEARMOE_OK) return rc;
    // 5. residual, grouped by expert (segments = the dispatch offsets)
    rc = residual_impl(s, A, z, perm, offsets, gate, P, Q, u, hres, st);
    if (rc != CLEARMOE_OK) return rc;
    // 6. y[t] = h_sh[t] + sum_j h_res[inv[t*k+j]]
    CLEARMOE_STAGE(CLEARMOE_STAGE_COMBINE_RES, st,
                   launch_combine_residual(s.dtype, hsh, hres, inv, y, T, s.D, s.k, A, st));
    // 7. class tokens: the dense FFN's output replaces theirs
    if (cls) return class_tokens_impl(s, *router, x, W1, b1, b2, z, true, y, L, ws, st);
    return CLEARMOE_OK;
}

}  // namespace

namespace {

// Copies [batches][rows][cols] of src into the workspace region at off as
// [batches][prow][pcol] with zeros around; a NULL src (an operand the path
// does not read) stays NULL.
int pad_operand(int eb, const void* src, void* ws, size_t off, int64_t batches, int64_t rows,
                int64_t cols, int64_t prow, int64_t pcol, hipStream_t st, const void** out) {
    *out = nullptr;
    if (src == nullptr) return CLEARMOE_OK;
    void* dst = at<void>(ws, off);
    if (launch_pad_copy(eb, src, dst, batches, rows, cols, prow, pcol, st) != hipSuccess)
        return CLEARMOE_ERR_HIP;
    *out = dst;
    return CLEARMOE_OK;
}

bool elem_aligned(const void* p, size_t a) { return p == nullptr || aligned(p, a); }

// The layer on an unaligned shape: padded copies of its operands, the
// aligned layer on them, y cropped back (see pad_layout).  Operands are read
// element by element, so element alignment suffices.
int ffn_forward_unaligned(const clearmoe_shape& s, const clearmoe_router* router, const void* x,
                          const void* W1, const float* b1, const void* US, const void* Vt,
                          const float* b2, const void* P, const void* Q, void* y, int32_t* idx_out,
                          float* gate_out, void* ws, size_t ws_bytes, hipStream_t st) {
    const size_t es = elem_size(s.dtype);
    if (router == nullptr || router->Wg == nullptr || !W1 || (s.T > 0 && (!x || !y)))
        return CLEARMOE_ERR_INVALID_ARG;
    if ((s.r > 0 && (!US || !Vt)) || (s.q > 0 && (!P || !Q))) return CLEARMOE_ERR_INVALID_ARG;
    if (router->hidden < 0 || router->hidden > kMlpHiddenMax || (router->hidden > 0 && !router->Wh))
        return CLEARMOE_ERR_INVALID_ARG;
    const void* ve[] = {x, W1, US, Vt, P, Q, y, router->Wg, router->Wh, router->W2};
    for (const void* p : ve)
        if (!elem_aligned(p, es)) return CLEARMOE_ERR_INVALID_ARG;
    const void* v4[] = {b1, b2, idx_out, gate_out};
    for (const void* p : v4)
        if (!elem_aligned(p, 4)) return CLEARMOE_ERR_INVALID_ARG;
    const PadLayout pl = pad_layout(s);
    if (!ws || !aligned(ws, kAlign) || ws_bytes < pl.total) return CLEARMOE_ERR_WORKSPACE;
    const clearmoe_shape a = aligned_shape(s);
    const int eb = static_cast<int>(es);
    const int64_t T = s.T, E = s.E;
    const void *xp, *W1p, *b1p, *USp, *Vtp, *b2p, *Pp, *Qp;
    int rc = pad_operand(eb, x, ws, pl.x, 1, T, s.D, T, a.D, st, &xp);
    if (rc == CLEARMOE_OK) rc = pad_operand(eb, W1, ws, pl.W1, 1, s.H, s.D, a.H, a.D, st, &W1p);
    if (rc == CLEARMOE_OK) rc = pad_operand(4, b1, ws, pl.b1, 1, 1, s.H, 1, a.H, st, &b1p);
    if (rc == CLEARMOE_OK) rc = pad_operand(eb, s.r > 0 ? US : nullptr, ws, pl.US, 1, s.D, s.r, a.D, a.r, st, &USp);
    if (rc == CLEARMOE_OK) rc = pad_operand(eb, s.r > 0 ? Vt : nullptr, ws, pl.Vt, 1, s.r, s.H, a.r, a.H, st, &Vtp);
    if (rc == CLEARMOE_OK) rc = pad_operand(4, b2, ws, pl.b2, 1, 1, s.D, 1, a.D, st, &b2p);
    if (rc == CLEARMOE_OK) rc = pad_operand(eb, s.q > 0 ? P : nullptr, ws, pl.P, E, s.D, s.q, a.D, a.q, st, &Pp);
    if (rc == CLEARMOE_OK) rc = pad_operand(eb, s.q > 0 ? Q : nullptr, ws, pl.Q, E, s.q, s.H, a.q, a.H, st, &Qp);
    clearmoe_router rt = *router;
    if (rc == CLEARMOE_OK && rt.hidden == 0)   // linear router: Wg [E, D]
        rc = pad_operand(eb, router->Wg, ws, pl.Wg, 1, E, s.D, E, a.D, st, &rt.Wg);
    if (rc == CLEARMOE_OK && rt.hidden > 0)    // MLP router: Wh [hidden, D] (Wg is [E, hidden])
        rc = pad_operand(eb, router->Wh, ws, pl.Wh, 1, rt.hidden, s.D, rt.hidden, a.D, st, &rt.Wh);
    if (rc == CLEARMOE_OK && rt.W2 != nullptr)  // class tokens' fc2 [D, H]
        rc = pad_operand(eb, router->W2, ws, pl.W2, 1, s.D, s.H, a.D, a.H, st, &rt.W2);
    if (rc != CLEARMOE_OK) return rc;
    void* yp = at<void>(ws, pl.y);
    rc = ffn_forward_impl(&a, &rt, xp, W1p, static_cast<const float*>(b1p), USp, Vtp,
                          static_cast<const float*>(b2p), Pp, Qp, yp, idx_out, gate_out,
                          at<void>(ws, pl.inner), layout(a).total, st);
    if (rc != CLEARMOE_OK || T == 0) return rc;
    return launch_pad_copy(eb, yp, y, 1, T, a.D, T, s.D, st) == hipSuccess ? CLEARMOE_OK : CLEARMOE_ERR_HIP;
}

// Routing on padded copies (see route_pads).  The router has been checked
// with element alignment; x too is read element by element.
int route_unaligned(const clearmoe_shape& s, const clearmoe_router& router, const void* x,
                    int32_t* idx, float* gate, void* ws, size_t ws_bytes, hipStream_t st) {
    const size_t es = elem_size(s.dtype);
    if (router.Wg == nullptr || (s.T > 0 && (!x || !idx || !gate))) return CLEARMOE_ERR_INVALID_ARG;
    if (!elem_aligned(x, es) || !elem_aligned(router.Wg, es) || !elem_aligned(idx, 4) ||
        !elem_aligned(gate, 4) || !elem_aligned(router.bg, 4))
        return CLEARMOE_ERR_INVALID_ARG;
    const RoutePads rp = route_pads(s);
    if (!ws || !aligned(ws, kAlign) || ws_bytes < rp.total) return CLEARMOE_ERR_WORKSPACE;
    const int eb = static_cast<int>(es);
    const int64_t T = s.T, E = s.E;
    const void* xp;
    int rc = pad_operand(eb, x, ws, rp.x, 1, T, s.D, T, rp.a.D, st, &xp);
    clearmoe_router rt = router;
    if (rc == CLEARMOE_OK && rt.hidden == 0)   // linear router: Wg [E, D]
        rc = pad_operand(eb, router.Wg, ws, rp.Wg, 1, E, s.D, E, rp.a.D, st, &rt.Wg);
    if (rc == CLEARMOE_OK && rt.hidden > 0)    // MLP router: Wh [hidden, D] (Wg is [E, hidden])
        rc = pad_operand(eb, router.Wh, ws, rp.Wh, 1, rt.hidden, s.D, rt.hidden, rp.a.D, st, &rt.Wh);
    if (rc != CLEARMOE_OK) return rc;
    return route_impl(rp.a, layout(rp.a), rt, xp, idx, gate, ws, st);
}

// Layer entry: unaligned shapes through the padded copies, others directly.
int ffn_forward_any(const clearmoe_shape* shape, const clearmoe_router* router, const void* x,
                    const void* W1, const float* b1, const void* US, const void* Vt, const float* b2,
                    const void* P, const void* Q, void* y, int32_t* idx_out, float* gate_out, void* ws,
                    size_t ws_bytes, hipStream_t st) {
    if (shape != nullptr && check_shape(shape, true, true) == CLEARMOE_OK && unaligned_layer(*shape))
        return ffn_forward_unaligned(*shape, router, x, W1, b1, US, Vt, b2, P, Q, y, idx_out, gate_out,
                                     ws, ws_bytes, st);
    return ffn_forward_impl(shape, router, x, W1, b1, US, Vt, b2, P, Q, y, idx_out, gate_out, ws, ws_bytes,
                            st);
}

}  // namespace

extern "C" {

int clearmoe_ffn_forward(const clearmoe_shape* shape, const void* x, const void* W1,
                         const float* b1, const void* US, const void* Vt, const float* b2,
                         const void* P, const void* Q, const void* Wg, const float* bg, void* y,
                         int32_t* idx_out, float* gate_out, void* ws, size_t ws_bytes,
                         hipStream_t stream) {
    const clearmoe_router rt = linear_router(Wg, bg);
    return ffn_forward_any(shape, &rt, x, W1, b1, US, Vt, b2, P, Q, y, idx_out, gate_out, ws, ws_bytes,
                           stream);
}

}  // extern "C"

namespace {

// Scratch of clearmoe_ffn_forward_noalloc: one fixed device array, which each
// device the library runs on holds until the process ends.  In host code the
// name `scratch` only stands for the symbol: its device address on the
// current device comes from hipGetSymbolAddress, once per device, and only
// that address is handed to kernels.
static __device__ __align__(256) unsigned char scratch[CLEARMOE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch` (looked up on the first call on
// that device, with it current).
int scratch_address(void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return CLEARMOE_ERR_HIP;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
            return CLEARMOE_ERR_HIP;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return CLEARMOE_OK;
}

}  // namespace

extern "C" {

int clearmoe_ffn_forward_noalloc(const clearmoe_shape* shape, const void* x, const void* W1,
                                 const float* b1, const void* US, const void* Vt, const float* b2,
                                 const void* P, const void* Q, const void* Wg, const float* bg,
                                 void* y, int32_t* idx_out, float* gate_out, hipStream_t stream) {
    int rc = check_layer_args(shape, x, W1, b1, US, Vt, b2, P, Q, Wg, bg, y, idx_out, gate_out);
    if (rc != CLEARMOE_OK) return rc;
    const Layout L = layout_min(*shape);
    if (L.total > static_cast<size_t>(CLEARMOE_NOALLOC_SCRATCH_BYTES)) return CLEARMOE_ERR_TOO_LARGE;
    void* ws = nullptr;
    rc = scratch_address(&ws);
    if (rc != CLEARMOE_OK) return rc;
    const clearmoe_router rt = linear_router(Wg, bg);
    return ffn_forward_impl(shape, &rt, x, W1, b1, US, Vt, b2, P, Q, y, idx_out, gate_out, ws,
                            L.total, stream, &L);
}

int clearmoe_ffn_forward_ex(const clearmoe_shape* shape, const clearmoe_router* router,
                            const void* x, const void* W1, const float* b1, const void* US,
                            const void* Vt, const float* b2, const void* P, const void* Q,
                            void* y, int32_t* idx_out, float* gate_out, void* ws,
                            size_t ws_bytes, hipStream_t stream) {
    return ffn_forward_any(shape, router, x, W1, b1, US, Vt, b2, P, Q, y, idx_out, gate_out, ws, ws_bytes,
                           stream);
}

size_t clearmoe_padded_workspace_bytes(const clearmoe_shape* shape) {
    if (check_shape(shape, true) != CLEARMOE_OK) return 0;
    return layout(*shape).padded_total;
}

int clearmoe_ffn_forward_padded(const clearmoe_shape* shape, const void* x, const void* W1,
                                const float* b1, const void* US, const void* Vt, const float* b2,
                                const void* P, const void* Q, const void* Wg, const float* bg,
                                void* y, int32_t* idx_out, float* gate_out, void* ws,
                                size_t ws_bytes, hipStream_t stream) {
    int rc = check_layer_args(shape, x, W1, b1, US, Vt, b2, P, Q, Wg, bg, y, idx_out, gate_out);
    if (rc != CLEARMOE_OK) return rc;
    const clearmoe_shape& s = *shape;
    const clearmoe_router rt = linear_router(Wg, bg);
    rc = check_router(s, &rt);
    if (rc != CLEARMOE_OK) return rc;
    const Layout L = layout(s);
    if (!ws || !aligned(ws, kAlign) || ws_bytes < L.padded_total) return CLEARMOE_ERR_WORKSPACE;
    if (s.T == 0) return CLEARMOE_OK;

    hipStream_t st = stream;
    const int64_t T = s.T, A = T * s.k;
    int32_t* idx = idx_out ? idx_out : at<int32_t>(ws, L.idx);
    float* gate = gate_out ? gate_out : at<float>(ws, L.gate);
    int32_t* counts = at<int32_t>(ws, L.counts);
    int32_t* offsets = at<int32_t>(ws, L.offsets);
    int32_t* perm = at<int32_t>(ws, L.perm);
    int32_t* inv = at<int32_t>(ws, L.inv);
    int32_t* perm_pad = at<int32_t>(ws, L.perm_pad);
    int32_t* inv_pad = at<int32_t>(ws, L.inv_pad);
    int32_t* seg = at<int32_t>(ws, L.seg);
    float* hsh = at<float>(ws, L.hsh);
    float* hres_pad = at<float>(ws, L.hres_pad);

    rc = route_impl(s, L, rt, x, idx, gate, ws, st);
    if (rc != CLEARMOE_OK) return rc;
    rc = dispatch_impl(s, L, idx, ws, counts, offsets, perm, inv, nullptr, nullptr, true, st);
    if (rc != CLEARMOE_OK) return rc;
    // The batch height is the largest expert count, which the host needs to
    // size the batched launches: copy the counts out, and overlap the round
    // trip with the shared stages.
    if (t_host_counts == nullptr &&
        hipHostMalloc(reinterpret_cast<void**>(&t_host_counts), 64 * sizeof(int32_t)) !=
            hipSuccess) {
        t_host_counts = nullptr;
        return CLEARMOE_ERR_HIP;
    }
    hipEvent_t ready = nullptr;
    if (hipEventCreateWithFlags(&ready, hipEventDisableTiming) != hipSuccess)
        return CLEARMOE_ERR_HIP;
    struct EventGuard {
        hipEvent_t e;
        ~EventGuard() { (void)hipEventDestroy(e); }
    } guard{ready};
    if (hipMemcpyAsync(t_host_counts, counts, sizeof(int32_t) * s.E, hipMemcpyDeviceToHost, st) !=
            hipSuccess ||
        hipEventRecord(ready, st) != hipSuccess)
        return CLEARMOE_ERR_HIP;
    rc = shared_impl(s, x, W1, b1, US, Vt, b2, at<void>(ws, L.z), at<void>(ws, L.tproj), hsh, st);
    if (rc != CLEARMOE_OK) return rc;
    if (hipEventSynchronize(ready) != hipSuccess) return CLEARMOE_ERR_HIP;
    int64_t C = 0;
    for (int e = 0; e < s.E; ++e)
        if (t_host_counts[e] > C) C = t_host_counts[e];
    if (C < 1 || C > A) return CLEARMOE_ERR_HIP;   // counts sum to A > 0

    // E sub-batches of C rows each (padding rows gather nothing and are
    // carried through both products as zero rows)
    CLEARMOE_STAGE(CLEARMOE_STAGE_PAD_INDEX, st,
                   launch_pad_index(idx, counts, offsets, perm, inv, A, s.E, C, perm_pad, inv_pad,
                                    seg, st));
    const int64_t M = static_cast<int64_t>(s.E) * C;
    rc = residual_impl(s, M, at<void>(ws, L.z), perm_pad, seg, gate, P, Q, at<void>(ws, L.u_pad),
                       hres_pad, st);
    if (rc != CLEARMOE_OK) return rc;
    CLEARMOE_STAGE(CLEARMOE_STAGE_COMBINE_RES, st,
                   launch_combine_residual(s.dtype, hsh, hres_pad, inv_pad, y, T, s.D, s.k, M,
                                           st));
    return CLEARMOE_OK;
}

int clearmoe_dense_ffn_forward(const clearmoe_shape* shape, const void* x, const void* W1,
                               const float* b1, const void* W2, const float* b2, void* y,
                               void* ws, size_t ws_bytes, hipStream_t stream) {
    if (shape != nullptr && check_shape(shape, true, true) == CLEARMOE_OK && unaligned_layer(*shape)) {
        // padded copies, the aligned FFN on them, y cropped (see pad_layout)
        const clearmoe_shape& s = *shape;
        const size_t es = elem_size(s.dtype);
        if (!W1 || !W2 || (s.T > 0 && (!x || !y))) return CLEARMOE_ERR_INVALID_ARG;
        const void* ve[] = {x, W1, W2, y};
        for (const void* p : ve)
            if (!elem_aligned(p, es)) return CLEARMOE_ERR_INVALID_ARG;
        if (!elem_aligned(b1, 4) || !elem_aligned(b2, 4)) return CLEARMOE_ERR_INVALID_ARG;
        const PadLayout pl = pad_layout(s);
        if (!ws || !aligned(ws, kAlign) || ws_bytes < pl.total) return CLEARMOE_ERR_WORKSPACE;
        const clearmoe_shape a = aligned_shape(s);
        const int eb = static_cast<int>(es);
        const void *xp, *W1p, *b1p, *W2p, *b2p;
        int rc = pad_operand(eb, x, ws, pl.x, 1, s.T, s.D, s.T, a.D, stream, &xp);
        if (rc == CLEARMOE_OK) rc = pad_operand(eb, W1, ws, pl.W1, 1, s.H, s.D, a.H, a.D, stream, &W1p);
        if (rc == CLEARMOE_OK) rc = pad_operand(4, b1, ws, pl.b1, 1, 1, s.H, 1, a.H, stream, &b1p);
        if (rc == CLEARMOE_OK) rc = pad_operand(eb, W2, ws, pl.W2, 1, s.D, s.H, a.D, a.H, stream, &W2p);
        if (rc == CLEARMOE_OK) rc = pad_operand(4, b2, ws, pl.b2, 1, 1, s.D, 1, a.D, stream, &b2p);
        if (rc != CLEARMOE_OK) return rc;
        void* yp = at<void>(ws, pl.y);
        rc = clearmoe_dense_ffn_forward(&a, xp, W1p, static_cast<const float*>(b1p), W2p,
                                        static_cast<const float*>(b2p), yp, at<void>(ws, pl.inner),
                                        layout(a).total, stream);
        if (rc != CLEARMOE_OK || s.T == 0) return rc;
        return launch_pad_copy(eb, yp, y, 1, s.T, a.D, s.T, s.D, stream) == hipSuccess ? CLEARMOE_OK
                                                                                       : CLEARMOE_ERR_HIP;
    }
    int rc = check_shape(shape, true);
    if (rc != CLEARMOE_OK) return rc;
    const clearmoe_shape& s = *shape;
    if (!W1 || !W2 || (s.T > 0 && (!x || !y))) return CLEARMOE_ERR_INVALID_ARG;
    const void* v16[] = {x, W1, W2, y};
    for (const void* p : v16)
        if (p && !aligned(p, 16)) return CLEARMOE_ERR_INVALID_ARG;
    if ((b1 && !aligned(b1, 4)) || (b2 && !aligned(b2, 4))) return CLEARMOE_ERR_INVALID_ARG;
    // only z is used: a workspace sized for a CLEAR-MoE layer of the same
    // T, D, H serves as well
    const Layout L = layout(s);
    const size_t need = L.z + elem_size(s.dtype) * static_cast<size_t>(s.T) * static_cast<size_t>(s.H);
    if (!ws || !aligned(ws, kAlign) || ws_bytes < need) return CLEARMOE_ERR_WORKSPACE;
    if (s.T == 0) return CLEARMOE_OK;
    void* z = at<void>(ws, L.z);
    GemmDesc g = gemm_desc(s.T, s.H, s.D);
    g.A = x; g.lda = s.D;
    g.B = W1; g.ldb = s.D;
    g.C = z; g.ldc = s.H; g.c_f32 = 0;
    g.bias = b1; g.gelu = 1;
    CLEARMOE_STAGE(CLEARMOE_STAGE_FC1, stream, launch_gemm(s.dtype, g, stream));
    g = gemm_desc(s.T, s.D, s.H);
    g.A = z; g.lda = s.H;
    g.B = W2; g.ldb = s.H;
    g.C = y; g.ldc = s.D; g.c_f32 = 0;
    g.bias = b2;
    CLEARMOE_STAGE(CLEARMOE_STAGE_DENSE_FC2, stream, launch_gemm(s.dtype, g, stream));
    return CLEARMOE_OK;
}

}  // extern "C"

namespace {

// The dense FFN y = GELU(x W1^T + b1) W2^T + b2 with z in the workspace.
int dense_impl(const clearmoe_shape& s, const void* x, const void* W1, const float* b1,
               const void* W2, const float* b2, void* y, void* z, hipStream_t st) {
    GemmDesc g = gemm_desc(s.T, s.H, s.D);
    g.A = x; g.lda = s.D;
    g.B = W1; g.ldb = s.D;
    g.C = z; g.ldc = s.H; g.c_f32 = 0;
    g.bias = b1; g.gelu = 1;
    CLEARMOE_STAGE(CLEARMOE_STAGE_FC1, st, launch_gemm(s.dtype, g, st));
    g = gemm_desc(s.T, s.D, s.H);
    g.A = z; g.lda = s.H;
    g.B = W2; g.ldb = s.H;
    g.C = y; g.ldc = s.D; g.c_f32 = 0;
    g.bias = b2;
    CLEARMOE_STAGE(CLEARMOE_STAGE_DENSE_FC2, st, launch_gemm(s.dtype, g, st));
    return CLEARMOE_OK;
}

// The shape of stack layer l (the stack's shape with the layer's k).
clearmoe_shape stack_layer_shape(const clearmoe_shape& s, const clearmoe_stack_layer& L) {
    clearmoe_shape sl = s;
    sl.k = L.moe ? L.k : 1;
    return sl;
}

// Largest per-layer workspace of a stack (0 if a layer is invalid).
size_t stack_layer_bytes(const clearmoe_shape& s, const clearmoe_stack_layer* layers, int32_t n) {
    size_t most = 0;
    for (int32_t l = 0; l < n; ++l) {
        if (layers[l].moe != 0 && layers[l].moe != 1) return 0;
        const clearmoe_shape sl = stack_layer_shape(s, layers[l]);
        if (check_shape(&sl, true) != CLEARMOE_OK) return 0;
        const size_t b = layout(sl).total;
        if (b > most) most = b;
    }
    return up(most);
}

}  // namespace

extern "C" {

size_t clearmoe_stack_workspace_bytes(const clearmoe_shape* shape,
                                      const clearmoe_stack_layer* layers, int32_t n) {
    if (shape == nullptr || layers == nullptr || n < 1) return 0;
    const size_t most = stack_layer_bytes(*shape, layers, n);
    if (most == 0) return 0;
    const size_t act = up(elem_size(shape->dtype) * static_cast<size_t>(shape->T > 0 ? shape->T : 0) *
                          static_cast<size_t>(shape->D));
    return most + 3 * act;
}

int clearmoe_stack_forward(const clearmoe_shape* shape, const clearmoe_stack_layer* layers,
                           int32_t n, int32_t residual, const void* x, void* y, void* ws,
                           size_t ws_bytes, hipStream_t stream) {
    if (shape == nullptr || layers == nullptr || n < 1) return CLEARMOE_ERR_INVALID_ARG;
    if (residual != 0 && residual != 1) return CLEARMOE_ERR_INVALID_ARG;
    const clearmoe_shape& s = *shape;
    // every layer's arguments are checked before the first launch
    for (int32_t l = 0; l < n; ++l) {
        const clearmoe_stack_layer& L = layers[l];
        if (L.moe != 0 && L.moe != 1) return CLEARMOE_ERR_INVALID_ARG;
        const clearmoe_shape sl = stack_layer_shape(s, L);
        int rc;
        if (L.moe) {
            rc = check_layer_args(&sl, x, L.W1, L.b1, L.US, L.Vt, L.b2, L.P, L.Q, nullptr, nullptr,
                                  y, nullptr, nullptr);
            if (rc == CLEARMOE_OK) rc = check_router(sl, &L.router);
            if (rc == CLEARMOE_OK && L.router.dense_stride > 0 && L.router.W2 == nullptr)
                rc = CLEARMOE_ERR_INVALID_ARG;
        } else {
            rc = check_shape(&sl, true);
            if (rc == CLEARMOE_OK && (!L.W1 || !L.W2 || !aligned(L.W1, 16) || !aligned(L.W2, 16) ||
                                      (L.b1 && !aligned(L.b1, 4)) || (L.b2 && !aligned(L.b2, 4))))
                rc = CLEARMOE_ERR_INVALID_ARG;
        }
        if (rc != CLEARMOE_OK) return rc;
    }
    if (s.T > 0 && (!x || !y || !aligned(x, 16) || !aligned(y, 16))) return CLEARMOE_ERR_INVALID_ARG;
    const size_t need = clearmoe_stack_workspace_bytes(shape, layers, n);
    if (need == 0) return CLEARMOE_ERR_INVALID_ARG;
    if (!ws || !aligned(ws, kAlign) || ws_bytes < need) return CLEARMOE_ERR_WORKSPACE;
    if (s.T == 0) return CLEARMOE_OK;

    // workspace: the layers' own region first, then activations A, B and the
    // layer output F
    const size_t most = stack_layer_bytes(s, layers, n);
    const size_t act = up(elem_size(s.dtype) * static_cast<size_t>(s.T) * static_cast<size_t>(s.D));
    void* buf[2] = {at<void>(ws, most), at<void>(ws, most + act)};
    void* F = at<void>(ws, most + 2 * act);
    const void* cur = x;
    for (int32_t l = 0; l < n; ++l) {
        const clearmoe_stack_layer& L = layers[l];
        const clearmoe_shape sl = stack_layer_shape(s, L);
        void* out = l == n - 1 ? y : buf[l % 2];
        void* f = residual ? F : out;
        int rc;
        if (L.moe) {
            rc = ffn_forward_impl(&sl, &L.router, cur, L.W1, L.b1, L.US, L.Vt, L.b2, L.P, L.Q, f,
                                  nullptr, nullptr, ws, most, stream);
        } else {
            rc = dense_impl(sl, cur, L.W1, L.b1, L.W2, L.b2, f, at<void>(ws, layout(sl).z), stream);
        }
        if (rc != CLEARMOE_OK) return rc;
        if (residual)
            CLEARMOE_STAGE(CLEARMOE_STAGE_RESIDUAL_ADD, stream,
                           launch_residual_add(s.dtype, cur, F, out, s.T, s.D, stream));
        cur = out;
    }
    return CLEARMOE_OK;
}

const char* clearmoe_stage_name(int stage) {
    static const char* names[CLEARMOE_N_STAGES] = {
        "route", "tile_hist", "scan", "permute", "combine", "fc1_gelu",
        "basis_t", "basis_h", "res_u", "res_h", "combine_res", "dense_fc2", "tu_grouped",
        "y_grouped", "fused_top1", "pad_index", "pair_key", "tu_pair", "y_pair",
        "residual_add"};
    return (stage >= 0 && stage < CLEARMOE_N_STAGES) ? names[stage] : "?";
}

int clearmoe_timing_start(unsigned stage_mask, int max_records) {
    return clearmoe_timing_start_sampled(stage_mask, max_records, 1);
}

int clearmoe_timing_start_sampled(unsigned stage_mask, int max_records, int every) {
    std::lock_guard<std::mutex> lk(g_timer_mu);
    if (g_timer.on || max_records < 1 || every < 1) return CLEARMOE_ERR_INVALID_ARG;
    g_timer.ev.assign(2 * static_cast<size_t>(max_records), nullptr);
    g_timer.stage.assign(static_cast<size_t>(max_records), -1);
    for (auto& e : g_timer.ev) {
        if (hipEventCreate(&e) != hipSuccess) {
            for (auto& f : g_timer.ev)
                if (f) (void)hipEventDestroy(f);
            g_timer.ev.clear();
            g_timer.stage.clear();
            return CLEARMOE_ERR_HIP;
        }
    }
    g_timer.mask = stage_mask;
    g_timer.used = 0;
    g_timer.every = every;
    g_timer.seen = 0;
    g_timer.on = true;
    return CLEARMOE_OK;
}

int clearmoe_timing_stop(double* ms, int32_t* launches) {
    std::lock_guard<std::mutex> lk(g_timer_mu);
    if (!g_timer.on) return CLEARMOE_ERR_INVALID_ARG;
    double acc[CLEARMOE_N_STAGES] = {};
    int32_t cnt[CLEARMOE_N_STAGES] = {};
    int rc = CLEARMOE_OK;
    for (int i = 0; i < g_timer.used; ++i) {
        if (g_timer.stage[i] < 0) continue;   // the stage launched no kernel
        float t = 0.0f;
        if (hipEventSynchronize(g_timer.ev[2 * i + 1]) != hipSuccess ||
            hipEventElapsedTime(&t, g_timer.ev[2 * i], g_timer.ev[2 * i + 1]) != hipSuccess) {
            rc = CLEARMOE_ERR_HIP;
            continue;
        }
        acc[g_timer.stage[i]] += t;
        cnt[g_timer.stage[i]] += 1;
    }
    for (auto& e : g_timer.ev) (void)hipEventDestroy(e);
    g_timer.ev.clear();
    g_timer.stage.clear();
    g_timer.on = false;
    for (int i = 0; i < CLEARMOE_N_STAGES; ++i) {
        if (ms) ms[i] = acc[i];
        if (launches) launches[i] = cnt[i];
    }
    return rc;
}

}  // extern "C"
