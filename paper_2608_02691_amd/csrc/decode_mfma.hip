// Matrix-core split-context decode scan (placeholder until the MFMA kernel lands).
#include "common.h"
#include "kernels.h"

namespace int2kv {

bool mfma_decode_available() { return false; }

size_t qop_bytes(int B, int H, int gq) {
  (void)B;
  (void)H;
  (void)gq;
  return 0;
}

hipError_t launch_decode_split_mfma(const DecodeArgs& a, hipStream_t s) {
  (void)a;
  (void)s;
  return hipErrorNotSupported;
}

}  // namespace int2kv
