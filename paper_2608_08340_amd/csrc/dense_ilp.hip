// The top-5 list instances of the dense scoring kernel (OPRAG_ILP_KERNELS in dense.hip),
// compiled on their own so that the build can give this file the instruction-level-parallelism
// machine scheduler: the rest of dense.hip is left out here.
#define OPRAG_DENSE_ILP
#include "dense.hip"
