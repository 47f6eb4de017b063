// Kernel instantiations for stage count 11.
#include "poseidon_inst.h"

namespace pk {

PK_INST(11)

}  // namespace pk
