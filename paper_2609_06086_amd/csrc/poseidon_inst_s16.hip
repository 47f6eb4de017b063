// Kernel instantiations for stage count 16.
#include "poseidon_inst.h"

namespace pk {

PK_INST(16)

}  // namespace pk
