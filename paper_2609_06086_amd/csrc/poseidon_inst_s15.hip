// Kernel instantiations for stage count 15.
#include "poseidon_inst.h"

namespace pk {

PK_INST(15)

}  // namespace pk
