// Instantiations of the fused top-1 kernel with the class rows' workgroups
// (k_fused_top1_cls, fused_kernel.h): a translation unit of their own so that
// they compile in parallel with the other two sets.
#include "fused_kernel.h"

namespace clearmoe {

hipError_t fused_launch_cls(const FusedArgs& a, const ClassArgs& c, size_t lds, int grid, int nft,
                            hipStream_t st) {
    switch (nft) {
        case 1: return fused_cfg_cls<1>(a, c, lds, grid, st);
        case 2: return fused_cfg_cls<2>(a, c, lds, grid, st);
        case 3: return fused_cfg_cls<3>(a, c, lds, grid, st);
        case 4: return fused_cfg_cls<4>(a, c, lds, grid, st);
        default: return fused_cfg_cls<5>(a, c, lds, grid, st);
    }
}

}  // namespace clearmoe
