// The segment-kernel classes: every (S, M) compiled, for each scoring mode.
#include "seg_kernel.h"
#include "wseg_kernel.h"

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
// Multi-wave segments: {waves, instances per lane}, after the one-wave ones.
#define RT_WSEG_SHAPE(W_, M_) {W_, M_},
const SegShape kWideShapes[] = {RT_WSEG_FOR_EACH(RT_WSEG_SHAPE)};
#undef RT_WSEG_SHAPE
constexpr int kNumWide = (int)(sizeof(kWideShapes) / sizeof(kWideShapes[0]));
constexpr int kModes[] = {kModeTrue, kModeProxy, kModeBase, kModeTrueSampled, kModeProxySampled};
constexpr int kNumModes = (int)(sizeof(kModes) / sizeof(kModes[0]));

// Batched-service shapes {S, M}: the segment ones (one instance per lane
// first, then two), then the general one-replica-per-lane class {1, 0}.
#define RT_BSEG_SHAPE(S_, M_) {S_, M_},
const SegShape kBatShapes[] = {RT_BSEG_FOR_EACH(RT_BSEG_SHAPE){1, 0}};
#undef RT_BSEG_SHAPE
constexpr int kNumBat = (int)(sizeof(kBatShapes) / sizeof(kBatShapes[0]));

}  // namespace

// The one-wave and multi-wave classes of every mode, then the batched
// service model's classes (one replica per lane; their launch is
// launch_bat).
int sim_class_count() { return (kNumShapes + kNumWide) * kNumModes + kNumBat; }

SimClass sim_class(int i) {
  if (i >= (kNumShapes + kNumWide) * kNumModes) {
    const SegShape& e = kBatShapes[i - (kNumShapes + kNumWide) * kNumModes];
    return SimClass{kBat, e.S, e.M, e.M, kModeTrue};
  }
  if (i < kNumShapes * kNumModes) {
    const SegShape& e = kShapes[i % kNumShapes];
    return SimClass{kSeg, e.S, e.M, e.M, kModes[i / kNumShapes]};
  }
  i -= kNumShapes * kNumModes;
  const SegShape& e = kWideShapes[i % kNumWide];
  return SimClass{kWseg, 64 * e.S, e.M, e.M, kModes[i / kNumWide]};
}

hipError_t launch_sim(const SimClass& c, const SimArgs& a, hipStream_t stream) {
  if (c.kind == kBat) return hipErrorInvalidValue;  // needs its scratch: launch_bat
  const bool w = c.kind == kWseg;
  const int S = w ? c.S / 64 : c.S;
  switch (c.mode) {
    case kModeTrue:
      return w ? seg::launch_wide_mode<kModeTrue>(S, c.MP, a, stream) : seg::launch_mode<kModeTrue>(S, c.MP, a, stream);
    case kModeProxy:
      return w ? seg::launch_wide_mode<kModeProxy>(S, c.MP, a, stream)
               : seg::launch_mode<kModeProxy>(S, c.MP, a, stream);
    case kModeBase:
      return w ? seg::launch_wide_mode<kModeBase>(S, c.MP, a, stream) : seg::launch_mode<kModeBase>(S, c.MP, a, stream);
    case kModeTrueSampled:
      return w ? seg::launch_wide_mode<kModeTrueSampled>(S, c.MP, a, stream)
               : seg::launch_mode<kModeTrueSampled>(S, c.MP, a, stream);
    case kModeProxySampled:
      return w ? seg::launch_wide_mode<kModeProxySampled>(S, c.MP, a, stream)
               : seg::launch_mode<kModeProxySampled>(S, c.MP, a, stream);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace rt
