// Segment-kernel and wide-segment-kernel instances for the base scoring
// mode (one source file per mode, so that they compile in parallel).
#include "seg_kernel.h"
#include "wseg_kernel.h"

namespace rt {
namespace seg {

#define RT_SEG_CASE(S_, M_) \
  if (S == S_ && M == M_) return launch_seg<S_, M_, kModeBase>(a, stream);

template <>
hipError_t launch_mode<kModeBase>(int S, int M, const SimArgs& a, hipStream_t stream) {
  RT_SEG_FOR_EACH(RT_SEG_CASE)
  return hipErrorInvalidValue;
}

#define RT_WSEG_CASE(W_, M_) \
  if (W == W_ && M == M_) return launch_wseg<W_, M_, kModeBase>(a, stream);

template <>
hipError_t launch_wide_mode<kModeBase>(int W, int M, const SimArgs& a, hipStream_t stream) {
  RT_WSEG_FOR_EACH(RT_WSEG_CASE)
  return hipErrorInvalidValue;
}

}  // namespace seg
}  // namespace rt
