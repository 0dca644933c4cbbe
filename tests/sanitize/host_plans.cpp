// Host-only driver for the sanitizer test: the plans and the argument checks
// of libgbla.so (gbla_plan.cpp, gbla_ext_plan.cpp, gbla_api.cpp), built with
// -fsanitize=address,undefined and the kernel launchers replaced by stubs
// that only count their calls.  Every shape below goes through the plan and
// workspace arithmetic; an overflow, out-of-bounds access or other undefined
// behaviour aborts the run.  Prints "host plans ok" at the end.
#include <limits.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "gbla.h"
#include "gbla_ext.h"
#include "gbla_plan.h"

#define REQUIRE(cond)                                                          \
  do {                                                                         \
    if (!(cond)) {                                                             \
      fprintf(stderr, "host_plans: %s failed at line %d\n", #cond, __LINE__); \
      abort();                                                                 \
    }                                                                          \
  } while (0)

namespace gbla {
static int g_launches = 0;
gbla_status launch_conv(const Plan&, const void*, const void*, const void*, const float*,
                        const int32_t*, float*, float*, float*, hipStream_t) { ++g_launches; return GBLA_OK; }
gbla_status launch_state(const Plan& p, const void*, const void*, const void*, const float*,
                         const int32_t*, void*, float*, float*, float*, hipStream_t) {
  // the state and combine grids the real launcher builds
  REQUIRE(p.units >= 1 && p.heads >= 1 && (int64_t)p.nseq * p.heads <= INT32_MAX);
  ++g_launches;
  return GBLA_OK;
}
gbla_status launch_readout(const Plan& p, const void*, const void*, const float*, const float*,
                           const int32_t*, const void*, float*, hipStream_t, KernelEvents) {
  REQUIRE(p.runits >= 1 && p.heads >= 1);
  ++g_launches;
  return GBLA_OK;
}
gbla_status launch_backward(const Plan&, const BwdLayout&, const void*, const void*, const void*,
                            const void*, const void*, const float*, const float*, const int32_t*,
                            const float*, void*, float*, float*, float*, float*, float*, float*,
                            float*, hipStream_t) { ++g_launches; return GBLA_OK; }
gbla_status launch_project(const LayerPlan&, const void*, const float*, const void*,
                           const int32_t*, void*, void*, void*, void*, void*, void*, hipStream_t) {
  ++g_launches;
  return GBLA_OK;
}
}  // namespace gbla

extern "C" hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }

namespace {

// Stand-in device pointers: aligned, never dereferenced by host code.
alignas(256) unsigned char g_buf[1024];
void* A() { return g_buf; }
const float* F() { return reinterpret_cast<const float*>(g_buf); }
float* FO() { return reinterpret_cast<float*>(g_buf); }
const int32_t* CU() { return reinterpret_cast<const int32_t*>(g_buf); }

gbla_shape shape(int32_t B, int32_t H, int32_t n, int32_t d, int32_t W = 4, int32_t msl = 0,
                 int32_t dtype = GBLA_BF16, uint32_t flags = 0) {
  gbla_shape s;
  s.batch = B;
  s.heads = H;
  s.seqlen = n;
  s.head_dim = d;
  s.conv_width = W;
  s.max_seqlen = msl;
  s.dtype = dtype;
  s.eps = 1e-6f;
  s.flags = flags;
  return s;
}

void drive(const gbla_shape& s) {
  fprintf(stderr, "shape B=%d H=%d n=%d d=%d W=%d max=%d dtype=%d flags=%u\n", s.batch, s.heads,
          s.seqlen, s.head_dim, s.conv_width, s.max_seqlen, s.dtype, s.flags);
  const size_t fwd = gbla_workspace_bytes(&s);
  const size_t bwd = gbla_backward_workspace_bytes(&s);
  for (int ragged = 0; ragged < 2; ++ragged) {
    gbla::Plan p;
    if (gbla::make_plan(&s, ragged != 0, &p) == GBLA_OK) {
      REQUIRE(p.total_bytes <= fwd);  // the workspace size covers both readings
      gbla::Plan b;
      if (gbla::backward_plan(p, &b) == GBLA_OK) {
        const gbla::BwdLayout L = gbla::make_bwd_layout(b);
        REQUIRE(L.total_bytes <= bwd);
      }
    }
  }
  // The entry points check everything and then call the (stubbed) launchers;
  // a workspace size of SIZE_MAX passes the size check, so the arithmetic
  // behind each launch runs too.
  const int32_t* cu_opts[2] = {nullptr, CU()};
  for (const int32_t* cu : cu_opts) {
    (void)gbla_forward(&s, A(), A(), A(), A(), A(), F(), F(), cu, A(), SIZE_MAX, FO(), nullptr);
    (void)gbla_state(&s, A(), A(), A(), F(), cu, A(), SIZE_MAX, FO(), FO(), nullptr);
    (void)gbla_readout(&s, A(), A(), F(), F(), cu, A(), SIZE_MAX, FO(), nullptr);
    (void)gbla_conv1d(&s, A(), A(), A(), F(), cu, FO(), FO(), FO(), nullptr);
    (void)gbla_backward(&s, A(), A(), A(), A(), A(), F(), F(), cu, F(), A(), SIZE_MAX, FO(), FO(),
                        FO(), FO(), FO(), FO(), FO(), nullptr);
  }
}

void drive_layer(int32_t B, int32_t L, int32_t dm, int32_t H, int32_t d, int32_t msl = 0) {
  gbla_layer_shape s;
  s.batch = B;
  s.seqlen = L;
  s.d_model = dm;
  s.heads = H;
  s.head_dim = d;
  s.conv_width = 4;
  s.max_seqlen = msl;
  s.dtype = GBLA_BF16;
  s.eps = 1e-6f;
  (void)gbla_layer_workspace_bytes(&s);
  const int32_t* cu_opts[2] = {nullptr, CU()};
  for (const int32_t* cu : cu_opts) {
    (void)gbla_layer_project(&s, A(), F(), A(), cu, A(), SIZE_MAX, A(), A(), A(), A(), A(), nullptr);
    (void)gbla_layer_forward(&s, A(), F(), A(), F(), cu, A(), SIZE_MAX, FO(), nullptr);
  }
}

}  // namespace

int main() {
  const int32_t dims[3] = {32, 64, 128};
  for (int32_t d : dims) {
    for (int32_t W = 1; W <= 4; ++W) drive(shape(1, 8, 32768, d, W));
    drive(shape(1, 1, INT32_MAX, d));           // the longest sequence an int32 can name
    drive(shape(1, 1, INT32_MAX - 1, d, 4, INT32_MAX));
    drive(shape(INT32_MAX, 1, 1, d));           // the most sequences
    drive(shape(1, 65535, 32768, d));           // the most heads
    drive(shape(2, 65535, INT32_MAX, d));
    drive(shape(64, 8, 0, d, 4, 0));            // ragged batch of empty sequences
    drive(shape(64, 8, 1, d, 4, 1));            // ragged batch with a single token
    drive(shape(1, 1, 1, d, 1, 1, GBLA_F32));
    drive(shape(8, 8, 2048, d, 4, 0, GBLA_F32, GBLA_BLA));
    drive(shape(8, 8, 2048, d, 4, 0, GBLA_BF16, GBLA_NO_GATE | GBLA_NO_NORM));
  }
  // invalid shapes are refused before any arithmetic
  drive(shape(0, 8, 1, 64));
  drive(shape(1, 0, 1, 64));
  drive(shape(1, 8, -1, 64));
  drive(shape(1, 65536, 1, 64));
  drive(shape(1, 8, 1, 48));
  drive(shape(1, 8, 1, 64, 5));
  drive(shape(1, 8, 1, 64, 4, -1));
  // layers: widest embeddings, most heads, longest sequences the 32-bit offsets allow
  drive_layer(8, 32768, 1024, 16, 64);
  drive_layer(1, 1, 16384, 1, 128);
  drive_layer(1, 65536, 16384, 4, 64);
  drive_layer(1, INT32_MAX, 64, 1, 32);
  drive_layer(64, 4096, 64, 65535, 32);
  drive_layer(3, 0, 1024, 16, 64, 0);
  drive_layer(3, 1, 1024, 16, 64, 1);
  drive_layer(1, 8, 16448, 4, 64);  // d_model beyond the supported range: refused
  printf("host plans ok (%d stub launches)\n", gbla::g_launches);
  return 0;
}
