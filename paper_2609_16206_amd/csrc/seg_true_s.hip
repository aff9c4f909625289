// Segment-kernel and wide-segment-kernel instances for the true scoring
// mode over two sampled candidates per pool (one source file per mode).
#include "seg_kernel.h"
#include "wseg_kernel.h"

namespace rt {
namespace seg {

#define RT_SEG_CASE(S_, M_) \
  if (S == S_ && M == M_) return launch_seg<S_, M_, kModeTrueSampled>(a, stream);

template <>
hipError_t launch_mode<kModeTrueSampled>(int S, int M, const SimArgs& a, hipStream_t stream) {
  RT_SEG_FOR_EACH(RT_SEG_CASE)
  return hipErrorInvalidValue;
}

#define RT_WSEG_CASE(W_, M_) \
  if (W == W_ && M == M_) return launch_wseg<W_, M_, kModeTrueSampled>(a, stream);

template <>
hipError_t launch_wide_mode<kModeTrueSampled>(int W, int M, const SimArgs& a, hipStream_t stream) {
  RT_WSEG_FOR_EACH(RT_WSEG_CASE)
  return hipErrorInvalidValue;
}

}  // namespace seg
}  // namespace rt
