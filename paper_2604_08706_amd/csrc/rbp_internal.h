// Internal helpers shared by the translation units of librbpolicy.so.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "rbpolicy.h"

namespace rbp {

// Thread-local error text (rbp_last_error); printf-style.
void set_error(const char* fmt, ...) __attribute__((format(printf, 1, 2)));
void clear_error();

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Workspace carving: sub-buffers aligned to 256 bytes.
struct WsCarver {
  uint8_t* base;
  size_t used = 0;
  explicit WsCarver(void* p) : base(static_cast<uint8_t*>(p)) {}
  template <class T>
  T* take(size_t count) {
    used = align_up(used, 256);
    T* p = reinterpret_cast<T*>(base ? base + used : nullptr);
    used += count * sizeof(T);
    return p;
  }
};

// Workspace layouts (byte counts; the same carving order is used at run time).
size_t sample_gather_ws(int64_t capacity);
size_t logprob_fwd_ws(int64_t T, int32_t V);
size_t loss_ws(int64_t T);
size_t loss_seq_ws(int64_t B);
size_t logprob_bwd_ws(int64_t Tc, int32_t d, int32_t V);
size_t fused_ws(int64_t Tc, int32_t d, int32_t V);
size_t note_use_ws(int64_t capacity);

// The two products of the log-prob backward for one chunk of Tn tokens, from
// dz^T (bf16 [round256(V)][ldGt], columns Tn..round256(Tn) zero):
// dhidden_c [Tn][d] overwritten (dh_half: fp32 [ldGt][d] scratch), dW [V][d]
// overwritten or accumulated.  Tn = 0 only zeroes dW (unless accumulating).
void launch_grad_products(const uint16_t* Hc, const uint16_t* W, const uint16_t* Gt,
                          int64_t ldGt, int64_t Tn, int32_t d, int32_t V, float* dhidden_c,
                          float* dh_half, float* dW, int accumulate, hipStream_t s);
// Its two parts: dW rows of the vocabulary tiles [tn_begin, tn_end) (256 rows
// each), and dhidden (with its split-K sum; row t scaled by cs[t] when cs is
// given).
// scratch (fp32, scratch_floats) may hold partial sums of dW's last round.
void launch_dweight(const uint16_t* Hc, const uint16_t* Gt, int64_t ldGt, int64_t Tn, int32_t d,
                    int32_t V, float* dW, int accumulate, int64_t tn_begin, int64_t tn_end,
                    hipStream_t s, float* scratch = nullptr, int64_t scratch_floats = 0);
void launch_dhidden(const uint16_t* W, const uint16_t* Gt, int64_t ldGt, int64_t Tn, int32_t d,
                    int32_t V, float* dhidden_c, float* dh_half, hipStream_t s,
                    const float* cs = nullptr);

}  // namespace rbp

#define RBP_REQUIRE(cond, code, ...)   \
  do {                                 \
    if (!(cond)) {                     \
      rbp::set_error(__VA_ARGS__);     \
      return (code);                   \
    }                                  \
  } while (0)

#define RBP_CHECK_LAUNCH(what)                                              \
  do {                                                                      \
    hipError_t e_ = hipGetLastError();                                      \
    if (e_ != hipSuccess) {                                                 \
      rbp::set_error("%s: %s", (what), hipGetErrorString(e_));              \
      return RBP_EHIP;                                                      \
    }                                                                       \
  } while (0)
