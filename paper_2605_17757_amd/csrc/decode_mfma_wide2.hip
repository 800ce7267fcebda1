// The split kernel's instances for 5 to 8 query heads per kv-head (two chunks of
// four heads in one wave), compiled apart from the others: this unit is built with
// the max-ilp instruction scheduler, which interleaves their score MFMAs and weight
// arithmetic better than the default, while the one-, three- and four-chunk
// instances would spill registers under it.  The kernel source is the same file.
#define OSCAR_SPLIT_TWO_CHUNK_UNIT
#include "decode_mfma.hip"
