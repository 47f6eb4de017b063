// Kernel instantiations for stage count 9.
#include "poseidon_inst.h"

namespace pk {

PK_INST(9)

}  // namespace pk
