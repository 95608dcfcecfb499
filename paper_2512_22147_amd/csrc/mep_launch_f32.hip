// fp32 instances of the streaming, column-reduce and fill kernels.
#define MEP_T float
#include "mep_launch.inc"
