// Thin-tile instances of the dX kernel: the tiles of a short last wave,
// each cut into feature halves and token parts (see thin_plan in
// kernels.hpp).  The kernel is the one in dx_bf16.hip; this unit
// instantiates only its thin forms, so that they compile in parallel with the
// whole-tile ones.
#define LORS_THIN_TILES 1
#include "dx_bf16.hip"
