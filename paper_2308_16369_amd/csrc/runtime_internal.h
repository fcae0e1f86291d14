// Host-side helpers shared between the sources of libsarathi's C-ABI.
#pragma once

#include <stddef.h>

#include "sarathi.h"

namespace sarathi {

// Every host-side check of sarathi_hybrid_layer_forward that does not
// involve the workspace (SARATHI_* error code, message set); on success
// *need = the workspace bytes the batch needs for this KV's max_seq_len
// (sarathi_workspace_layout(...).total).
int hybrid_check_noalloc(const sarathi_model_cfg* cfg, const sarathi_layer_weights* w, const sarathi_kv* kv,
                         int layer, const sarathi_hybrid_batch* batch, const void* x_in, const void* x_out,
                         size_t* need);

}  // namespace sarathi
