// Kernels and launchers of 1-word item sets (one compilation unit per item
// width, so the widths build in parallel).
#define EPIC_KERNEL_UNIT 1
#include "epic.hip"
