// spk_run_batch.hip -- the persistent step kernel's variants for batches of
// several steps of LIF neurons (binned delivery), in a translation unit of
// their own: the kernel source is spk_run.hip.
#define SPK_RUN_BATCH 1
#include "spk_run.hip"
