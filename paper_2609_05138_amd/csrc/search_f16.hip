// Kernels 1 and 3 of the fused BMU search over an fp16 codebook (the paper's
// storage precision, Sections 4.2 and 4.3): 512-neuron slices (8 neurons per lane, one
// 128-bit load per row), rows widened to fp32 once per load, fp32 sums.
#include "search_st.h"

namespace som {

hipError_t launch_search_k1_f16(const SearchArgs& a, hipStream_t stream) {
  if (a.K != 8) return hipErrorInvalidValue;
  switch (a.T) {
    case 1: return launch_tk<_Float16, 1, 8>(a, stream);
    case 2: return launch_tk<_Float16, 2, 8>(a, stream);
    case 4: return launch_tk<_Float16, 4, 8>(a, stream);
    case 8: return launch_tk<_Float16, 8, 8>(a, stream);
    case 16: return launch_tk<_Float16, 16, 8>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_search_st_f16(const SearchArgs& a, hipStream_t stream) {
  if (a.T != 8 || a.K != 8) return hipErrorInvalidValue;
  switch (a.group) {
    case 8: return launch_st<_Float16, 8, 8, 8>(a, stream);
    case 16: return launch_st<_Float16, 8, 8, 16>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace som
