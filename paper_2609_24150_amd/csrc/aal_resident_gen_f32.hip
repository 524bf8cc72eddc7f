// Register-resident schedule of the combined objectives: the instances for
// fp32 logits (the kernel is in aal_resident_gen.h).
#include "aal_resident_gen.h"

namespace aal {

hipError_t launch_general_resident_f32(const GenArgs& a, bool* used) { return launch_ti<F32>(a, used); }

}  // namespace aal
