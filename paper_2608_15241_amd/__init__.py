"""Mixed-adapter LoRA step with version-tagged paged attention on MI355X.

The computation lives in liblocal.so (HIP kernels for gfx950 behind the C ABI
of include/local.h). This package holds its sources, its build and a thin
ctypes binding with the same names as the C entry points.
"""
from .binding import (BLOCK_SIZE, EXPORTS, LIB_PATH, Call, KVManager, LocalError, Scheduler,
                      Workspace,
                      load_library, local_block_version_check, local_lora_grad,
                      local_lora_grad_grouped, local_lora_grad_input, local_lora_linear,
                      local_kv_pool_export, local_kv_pool_import,
                      local_lora_linear_grouped, local_paged_attn_decode,
                      local_paged_attn_decode_checked, local_paged_attn_decode_noalloc,
                      local_paged_attn_prefill, prepare_paged_attn_decode_checked,
                      prepare_block_version_check, prepare_paged_attn_decode_noalloc,
                      prepare_lora_grad, prepare_lora_grad_grouped, prepare_lora_grad_input,
                      prepare_lora_linear,
                      prepare_lora_linear_grouped,
                      prepare_paged_attn_decode, prepare_paged_attn_prefill)
