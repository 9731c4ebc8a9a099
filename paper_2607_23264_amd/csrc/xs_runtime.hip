// Host runtime helpers: status text, window validation, device attributes.
#include <cmath>

#include "xs_common.hpp"

extern "C" const char* xs_strerror(int code) {
  switch (code) {
    case XS_OK: return "ok";
    case XS_EINVAL: return "invalid argument";
    case XS_EUNSUPPORTED: return "unsupported shape or option";
    case XS_EHIP: return "HIP runtime or launch failure";
    case XS_EWORKSPACE: return "workspace missing or too small";
    case XS_ECAPACITY: return "a destination window exceeded its capacity";
    case XS_ETIMEOUT: return "a bounded dependency wait timed out";
    case XS_EBADINPUT: return "expert id out of range, or listed twice by one token";
    default: return "unknown status";
  }
}

extern "C" int xs_version(void) { return 100; }

namespace xs_host {

int make_winset(const xs_window* win, int32_t W, int64_t row_bytes, xs::WinSet* out) {
  if (!win || W < 1 || W > XS_MAX_WINDOWS || !out) return XS_EINVAL;
  out->n = W;
  for (int d = 0; d < XS_MAX_WINDOWS; ++d) {
    out->base[d] = nullptr;
    out->cap[d] = 0;
    out->stride[d] = 0;
    out->flag[d] = nullptr;
  }
  for (int d = 0; d < W; ++d) {
    const xs_window& w = win[d];
    if (!w.base || w.capacity_rows < 0) return XS_EINVAL;
    if (w.row_stride_bytes < row_bytes || (w.row_stride_bytes & 15) ||
        (reinterpret_cast<uintptr_t>(w.base) & 15))
      return XS_EINVAL;
    out->base[d] = static_cast<char*>(w.base);
    out->cap[d] = w.capacity_rows;
    out->stride[d] = w.row_stride_bytes;
    out->flag[d] = w.ready_flag;
  }
  return XS_OK;
}

int launch_status() { return hipGetLastError() == hipSuccess ? XS_OK : XS_EHIP; }

double wall_rate_hz() {
  int dev = 0, khz = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0.0;
  if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess) return 0.0;
  return 1000.0 * static_cast<double>(khz);
}

int num_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return n;
}

int64_t ns_to_ticks(int64_t ns) {
  if (ns <= 0) return 0;
  double r = wall_rate_hz();
  if (r <= 0) r = 1e8;
  return static_cast<int64_t>(std::ceil(static_cast<double>(ns) * r * 1e-9));
}

}  // namespace xs_host

extern "C" double xs_clock_rate_hz(void) { return xs_host::wall_rate_hz(); }
