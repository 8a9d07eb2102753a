// Entry points whose kernels are not built yet: they report UNSUPPORTED.
#include "common.h"

extern "C" {
int bc_block_workspace_size(const bc_block_desc*, size_t*) { return bc::fail(BC_ERR_UNSUPPORTED, "not built"); }
int bc_dit_block_forward(const bc_block_desc*, const bc_block_weights*, float*, float*, const float*, const void*,
                         void*, size_t, void*) { return bc::fail(BC_ERR_UNSUPPORTED, "not built"); }
int bc_model_create(const bc_model_desc*, const bc_model_weights*, bc_model**) { return bc::fail(BC_ERR_UNSUPPORTED, "not built"); }
int bc_model_destroy(bc_model*) { return BC_OK; }
int bc_sample_workspace_size(const bc_model*, int, size_t*) { return bc::fail(BC_ERR_UNSUPPORTED, "not built"); }
int bc_sample(const bc_model*, int, int, int, const uint8_t*, int, const bc_bary_params*, bc_cache_ring*, float*,
              const int64_t*, const void*, void*, size_t, void*) { return bc::fail(BC_ERR_UNSUPPORTED, "not built"); }
int bc_linear(int, int, int, const void*, const void*, const void*, void*, int, const float*, const float*, int, int,
              void*) { return bc::fail(BC_ERR_UNSUPPORTED, "not built"); }
int bc_attention(int, int, int, int, int, const void*, const void*, const void*, void*, int, void*, size_t, void*) {
    return bc::fail(BC_ERR_UNSUPPORTED, "not built");
}
int bc_attention_workspace_size(int, int, int, int, int, int, size_t*) { return bc::fail(BC_ERR_UNSUPPORTED, "not built"); }
}
