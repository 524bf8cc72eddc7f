// Register-resident schedule of the combined objectives: the instances for
// bf16 logits with an fp32 gradient (the kernel is in aal_resident_gen.h).
#include "aal_resident_gen.h"

namespace aal {

hipError_t launch_general_resident_bf16_g32(const GenArgs& a, bool* used) { return launch_tg<Bf16, GF32>(a, used); }

}  // namespace aal
