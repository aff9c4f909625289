// The segment-kernel classes: every (S, M) compiled, for each scoring mode.
#include "seg_kernel.h"

namespace rt {
namespace {

struct SegShape {
  int S, M;
};

#define RT_SEG_SHAPE(S_, M_) {S_, M_},
// Ordered by instances per lane, then segment width: the first class that
// holds a point has the shortest step (the choice when the replicas are too
// few to fill the GPU); a deeper lane packs more replicas per wave (the
// choice when there are many).
const SegShape kShapes[] = {RT_SEG_FOR_EACH(RT_SEG_SHAPE)};
#undef RT_SEG_SHAPE
constexpr int kNumShapes = (int)(sizeof(kShapes) / sizeof(kShapes[0]));
constexpr int kModes[] = {kModeTrue, kModeProxy, kModeBase};

}  // namespace

int seg_class_count() { return kNumShapes * 3; }

SimClass seg_class(int i) {
  const SegShape& e = kShapes[i % kNumShapes];
  return SimClass{kSeg, e.S, e.M, e.M, kModes[i / kNumShapes]};
}

hipError_t launch_seg_class(const SimClass& c, const SimArgs& a, hipStream_t stream) {
  switch (c.mode) {
    case kModeTrue:
      return seg::launch_mode<kModeTrue>(c.S, c.MP, a, stream);
    case kModeProxy:
      return seg::launch_mode<kModeProxy>(c.S, c.MP, a, stream);
    case kModeBase:
      return seg::launch_mode<kModeBase>(c.S, c.MP, a, stream);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace rt
