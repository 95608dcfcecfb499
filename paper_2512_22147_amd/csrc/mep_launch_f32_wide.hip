// fp32 instances of the wide streaming-kernel shapes.
#define MEP_T float
#define MEP_WIDE_TABLE
#include "mep_launch.inc"
