// Status strings and version of the PTD library.
#include "ptd_common.hpp"

extern "C" const char* ptd_status_string(int status) {
  switch (status) {
    case PTD_OK: return "ok";
    case PTD_ERR_NULL: return "a required pointer is NULL";
    case PTD_ERR_SHAPE: return "size out of range or inconsistent";
    case PTD_ERR_DTYPE: return "unsupported dtype";
    case PTD_ERR_ALIGN: return "misaligned pointer or leading dimension";
    case PTD_ERR_WORKSPACE: return "workspace missing or too small";
    case PTD_ERR_HIP: return "HIP runtime or launch failure";
    case PTD_ERR_BAD_TREE: return "malformed tree: parent[i] outside [-1, i)";
    case PTD_ERR_KV_LEN: return "kv_len < 0 or kv_len + T > L_cap";
    case PTD_ERR_BAD_PATH: return "accepted path: length outside [0, T] or node ids not strictly increasing in [0, T)";
    case PTD_ERR_PAGE: return "page id outside [0, num_pages)";
    case PTD_ERR_SCRATCH: return "problem needs more than the 64 MiB scratch of ptd_tree_attention_noalloc";
    default: return "unknown status";
  }
}

extern "C" int ptd_version(void) { return 100; }
