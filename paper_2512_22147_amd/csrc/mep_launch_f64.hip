// fp64 instances of the streaming, column-reduce and fill kernels.
#define MEP_T double
#include "mep_launch.inc"
