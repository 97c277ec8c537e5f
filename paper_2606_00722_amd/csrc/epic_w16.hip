// Kernels and launchers of 16-word item sets (one compilation unit per item
// width, so the widths build in parallel).
#define EPIC_KERNEL_UNIT 16
#include "epic.hip"
