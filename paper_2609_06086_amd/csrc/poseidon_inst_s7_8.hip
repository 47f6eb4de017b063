// Kernel instantiations for stage counts 7, 8.
#include "poseidon_inst.h"

namespace pk {

PK_INST(7) PK_INST(8)

}  // namespace pk
