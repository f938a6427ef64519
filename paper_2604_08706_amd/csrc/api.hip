// Status strings, thread-local error text and workspace sizing of the C ABI.

#include <cstdarg>
#include <cstdio>

#include "rbp_internal.h"

namespace {
thread_local char g_last_error[512] = "";
}

void rbp::set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
}

void rbp::clear_error() { g_last_error[0] = '\0'; }

extern "C" const char* rbp_last_error(void) { return g_last_error; }

extern "C" const char* rbp_status_string(int status) {
  switch (status) {
    case RBP_OK: return "ok";
    case RBP_EINVAL: return "invalid argument";
    case RBP_EUNSUPPORTED: return "unsupported shape";
    case RBP_EWORKSPACE: return "workspace too small";
    case RBP_EHIP: return "HIP launch failed";
    default: return "unknown status";
  }
}

extern "C" size_t rbp_workspace_bytes(int op, int64_t n, int32_t d, int32_t V) {
  switch (op) {
    case RBP_OP_SAMPLE_GATHER: return rbp::sample_gather_ws(n);
    case RBP_OP_LOGPROB_FWD: return rbp::logprob_fwd_ws(n, V < 1 ? 1 : V);
    case RBP_OP_LOSS: return rbp::loss_ws(n);
    case RBP_OP_LOGPROB_BWD: return rbp::logprob_bwd_ws(n, d, V < 1 ? 1 : V);
    case RBP_OP_LOSS_SEQ: return rbp::loss_seq_ws(n);
    case RBP_OP_FUSED: return rbp::fused_ws(n, d, V);
    case RBP_OP_NOTE_USE: return rbp::note_use_ws(n);
    default: return 0;
  }
}
