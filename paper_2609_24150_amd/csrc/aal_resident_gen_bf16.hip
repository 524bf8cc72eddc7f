// Register-resident schedule of the combined objectives: the instances for
// bf16 logits with a bf16 gradient (the kernel is in aal_resident_gen.h; the
// other input/gradient types are compiled in their own files so that the
// instances build in parallel).
#include "aal_resident_gen.h"

namespace aal {

hipError_t launch_general_resident_bf16(const GenArgs& a, bool* used) {
  if (a.gd == DType::kF32) return launch_general_resident_bf16_g32(a, used);
  return launch_tg<Bf16, GBf16>(a, used);
}


}  // namespace aal
