// Kernel instantiations for stage counts 1, 2, 3, 4.
#include "poseidon_inst.h"

namespace pk {

PK_INST(1) PK_INST(2) PK_INST(3) PK_INST(4)

}  // namespace pk
