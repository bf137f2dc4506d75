// The 256-wide register-resident bf16 kernel with 1 hidden layer (own
// compilation unit: the instantiations build in parallel).
#include "mlp_bf16r.hpp"

namespace hpacml {

HPACML_BF16R_H256_UNIT(1)

}  // namespace hpacml
