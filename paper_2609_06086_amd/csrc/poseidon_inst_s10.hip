// Kernel instantiations for stage count 10.
#include "poseidon_inst.h"

namespace pk {

PK_INST(10)

}  // namespace pk
