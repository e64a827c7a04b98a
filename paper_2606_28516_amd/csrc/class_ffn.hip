// Host side of the class tokens' dense FFN (class_ffn.h): the split plan and
// the standalone launch.
#include <atomic>

#include "class_ffn.h"

namespace clearmoe {

namespace {

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_class_ffn(ClassArgs c) {
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    class_ffn_block(c, blockIdx.x, lds);
}

// Launch numbers of the arrival words: distinct for every launch of the
// process (1, 2, ...; 2^48 launches before one comes back).
std::atomic<uint64_t> g_launch{0};

}  // namespace

bool class_ffn_supported(int D, int H) {
    // up to 6144 hidden units the LDS plan (z chunk and b1) stays within 32 KB
    return D >= 8 && D <= kClsMaxD && D % 8 == 0 && H >= 8 && H <= 6144 && H % 8 == 0;
}

int64_t class_ffn_plan(ClassArgs& c, float* part, uint64_t* count) {
    const int64_t blocks = class_blocks(c.ncls);
    const int nchunks = (c.H + kClsChunk - 1) / kClsChunk;
    // P parts per block while blocks x P stays near the chip's width and the
    // partial sums fit their region; then every part gets ceil(chunks / P)
    // chunks and P shrinks to the parts that have some
    int64_t P = kClsMaxParts;
    while (P > 1 && (blocks * P > 128 || blocks * P * kClsPartFloats * 4 > static_cast<int64_t>(kClsPartBytes) ||
                     blocks > kClsCountWords))
        P /= 2;
    if (P > nchunks) P = nchunks;
    const int per = static_cast<int>((nchunks + P - 1) / P);
    c.nparts = P > 1 ? (nchunks + per - 1) / per : 1;
    c.per = c.nparts > 1 ? per : nchunks;
    c.part = part;
    c.count = count;
    c.launch = (g_launch.fetch_add(1) + 1) & ((uint64_t{1} << 48) - 1);
    if (c.launch == 0) c.launch = g_launch.fetch_add(1) + 1;
    return blocks * c.nparts;
}

hipError_t launch_class_ffn(const ClassArgs& c, hipStream_t st) {
    if (!class_ffn_supported(c.D, c.H) || c.stride < 1 || c.ncls < 0 || c.nparts < 1) return hipErrorInvalidValue;
    if (c.ncls == 0) return hipSuccess;
    launch_kernel(k_class_ffn, dim3(static_cast<unsigned>(class_blocks(c.ncls) * c.nparts)), 256,
                  class_lds_bytes(c.H), st, c);
    return hipGetLastError();
}

}  // namespace clearmoe
