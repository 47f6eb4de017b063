// Kernel instantiations for stage count 13.
#include "poseidon_inst.h"

namespace pk {

PK_INST(13)

}  // namespace pk
