// Workgroup-to-task order of the attention launch. MI355X deals the workgroups
// of a launch round-robin over its 8 XCDs (workgroup L runs on XCD L % 8), each
// with its own L2. This order gives each XCD a contiguous run of the n tasks,
// so the tasks that stream the same key tiles (the Query blocks of one head)
// read them through one L2. It is a bijection of [0, n) for every n >= 1.
// Plain C so that a host test can check that.
#ifndef QWM_XCD_ORDER_H
#define QWM_XCD_ORDER_H

#include <stdint.h>

#ifdef __HIPCC__
#define QWM_HOST_DEVICE __host__ __device__
#else
#define QWM_HOST_DEVICE
#endif

static inline QWM_HOST_DEVICE uint32_t qwm_xcd_task(uint32_t L, uint32_t n) {
  const uint32_t P = L % 8, Q = L / 8, q = n / 8, rr = n % 8;
  // XCD P runs workgroups P, P + 8, ...: q + 1 of them when P < n % 8, else q
  return P < rr ? P * (q + 1) + Q : rr * (q + 1) + (P - rr) * q + Q;
}

#endif
