// Hidden-split instantiations of the fused top-1 kernel (fused_kernel.h): S
// workgroups per 64-row tile, each on every S-th group of hidden slices, for
// batches with fewer tiles than CUs.  A translation unit of its own so that
// the two sets of variants compile in parallel.
#include "fused_kernel.h"

namespace clearmoe {

hipError_t fused_launch_split(const FusedArgs& a, size_t lds, int grid, int nft, hipStream_t st) {
    switch (nft) {
        case 1: return fused_cfg<1, true>(a, lds, grid, st);
        case 2: return fused_cfg<2, true>(a, lds, grid, st);
        case 3: return fused_cfg<3, true>(a, lds, grid, st);
        case 4: return fused_cfg<4, true>(a, lds, grid, st);
        default: return fused_cfg<5, true>(a, lds, grid, st);
    }
}

}  // namespace clearmoe
