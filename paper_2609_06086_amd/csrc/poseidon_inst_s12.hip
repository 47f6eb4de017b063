// Kernel instantiations for stage count 12.
#include "poseidon_inst.h"

namespace pk {

PK_INST(12)

}  // namespace pk
