// Kernels and launchers of 8-word item sets (one compilation unit per item
// width, so the widths build in parallel).
#define EPIC_KERNEL_UNIT 8
#include "epic.hip"
