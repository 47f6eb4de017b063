// Kernel instantiations for stage counts 5, 6.
#include "poseidon_inst.h"

namespace pk {

PK_INST(5) PK_INST(6)

}  // namespace pk
