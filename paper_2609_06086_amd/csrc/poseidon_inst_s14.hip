// Kernel instantiations for stage count 14.
#include "poseidon_inst.h"

namespace pk {

PK_INST(14)

}  // namespace pk
