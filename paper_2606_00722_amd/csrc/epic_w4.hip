// Kernels and launchers of 4-word item sets (one compilation unit per item
// width, so the widths build in parallel).
#define EPIC_KERNEL_UNIT 4
#include "epic.hip"
