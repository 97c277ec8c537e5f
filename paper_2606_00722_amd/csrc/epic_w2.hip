// Kernels and launchers of 2-word item sets (one compilation unit per item
// width, so the widths build in parallel).
#define EPIC_KERNEL_UNIT 2
#include "epic.hip"
