// Shared host/device helpers of the gfx950 FastCHGNet library.
#pragma once
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>

#include "chgnet.h"

namespace chg {

// ---------------------------------------------------------------------------
// Error reporting: the last error text per host thread.
// ---------------------------------------------------------------------------
void set_error(const std::string& msg);
int fail(int code, const std::string& msg);

#define CHG_HIP(call)                                                                         \
  do {                                                                                        \
    hipError_t _e = (call);                                                                   \
    if (_e != hipSuccess)                                                                     \
      return ::chg::fail(CHGNET_EHIP, std::string(#call) + ": " + hipGetErrorString(_e));   \
  } while (0)

#define CHG_TRY(expr)           \
  do {                          \
    int _r = (expr);            \
    if (_r != CHGNET_OK) return _r; \
  } while (0)

// Launch-error check after a kernel launch.
#define CHG_LAUNCHED(name)                                                                    \
  do {                                                                                        \
    hipError_t _e = hipGetLastError();                                                        \
    if (_e != hipSuccess)                                                                     \
      return ::chg::fail(CHGNET_EHIP, std::string("launch ") + name + ": " + hipGetErrorString(_e)); \
  } while (0)

// Optional per-launch timing (measurement only; off unless enabled through
// chgnet_profile_start). Events bracket each launch on its own stream.
int prof_mark(hipStream_t st);                       // returns event index or -1
bool prof_active();
void prof_close(hipStream_t st, int first, const char* tag);

#define KLAUNCH(st, tag, ...)                                                                 \
  do {                                                                                        \
    const int _pf = ::chg::prof_mark(st);                                                     \
    __VA_ARGS__;                                                                              \
    hipError_t _e = hipGetLastError();                                                        \
    if (_e != hipSuccess)                                                                     \
      return ::chg::fail(CHGNET_EHIP, std::string("launch ") + (tag) + ": " + hipGetErrorString(_e)); \
    ::chg::prof_close(st, _pf, tag);                                                          \
  } while (0)

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Bump allocator over the caller's workspace (256-byte aligned slices).
struct Arena {
  char* base = nullptr;
  size_t cap = 0;
  size_t used = 0;
  template <class T>
  T* take(int64_t count) {
    size_t off = align_up(used, 256);
    used = off + sizeof(T) * (size_t)(count > 0 ? count : 0);
    if (base == nullptr || used > cap) return reinterpret_cast<T*>(base ? base + (off < cap ? off : 0) : nullptr);
    return reinterpret_cast<T*>(base + off);
  }
  bool ok() const { return used <= cap; }
};

int validate_hparams(const chgnet_hparams* hp);

// ---------------------------------------------------------------------------
// Flat parameter layout (see include/chgnet.h).
// ---------------------------------------------------------------------------
struct GatedOffsets {
  int64_t W, b, g_c, b_c, g_g, b_g;  // W [rows, 2d], b [2d], LayerNorm [d] x 4
};
struct LayerOffsets {
  GatedOffsets av;  // atom conv, W [3d, 2d]
  int64_t av_Wo, av_bo;
  GatedOffsets be;  // bond conv, W [4d, 2d]
  int64_t be_Wo, be_bo;
  GatedOffsets an;  // angle update (valid if has_angle), W [4d, 2d]
  bool has_angle;
};
struct HeadOffsets {
  int64_t W1, b1, W2, b2, W3, b3;
  int out;
};
constexpr int kMaxLayers = 16;
constexpr int kMaxTensors = 24 * kMaxLayers + 32;
struct ParamLayout {
  int64_t W_Z, f_a, f_b, W_e, b_e0, W_eb, W_th, b_th;
  LayerOffsets layer[kMaxLayers];
  HeadOffsets head[3];  // E, F, S
  int64_t M_W, M_b;     // magnetic-moment head (-1 without it)
  int64_t total;
  int ntensors;                 // every tensor in layout order
  int64_t toff[kMaxTensors], tlen[kMaxTensors];
};
// align = 1: the public flat layout; align = 4: every tensor starts on a
// 16-byte boundary (internal copy used for vector loads of the weights).
ParamLayout make_layout(const chgnet_hparams& hp, int align = 1);

}  // namespace chg
