// rv_fuse_accept_noalloc: the decision of rv_debug_fuse_accept for callers
// that cannot allocate device memory, with its scratch in a static device
// array instead of a cache's workspace.
//
// The scratch holds what the fusion/accept kernels write and read back within
// one call: per vocabulary chunk the softmax statistics of o, r and z and z's
// top-2 ([4][rows][nchunk][4] floats), then the merged log-sum-exps
// ([3][rows]), entropies ([2][rows]), argmaxes ([rows]) and decision margins
// ([batch][k+2]).  Fused rows and log-probabilities are not kept (the accept
// kernel recomputes the few fused values it needs from o and r, bit for bit),
// and no id history is written.  Every entry a call reads was written earlier
// in the same call, so nothing has to start at zero.
#include <mutex>

#include "rv_internal.h"

namespace {

constexpr int kChunk = 2048;                 // vocabulary chunk of the tail kernels
constexpr size_t kScratchBytes = (size_t)RV_NOALLOC_SCRATCH_BYTES;
constexpr size_t kMaxChunkRows = 65536;      // rows x chunks of the per-chunk statistics

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch` on each GPU, once looked up

// Address of this GPU's copy of the array (looked up once per device, with
// that device current).
rv_status scratch_on_current_device(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return rv_fail(RV_E_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return rv_fail(RV_E_STATE, "device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return rv_fail(RV_E_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return RV_OK;
}

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

}  // namespace

extern "C" rv_status rv_fuse_accept_noalloc(const float* d_logits, int32_t batch, int32_t k, int32_t vocab,
                                            const int32_t* d_draft_ids, const rv_fusion* fusion,
                                            int32_t* d_accept_len, int32_t* d_next_id, void* stream) {
  if (!d_logits || !fusion || !d_accept_len || !d_next_id)
    return rv_fail(RV_E_ARG, "logits, fusion and outputs must not be NULL");
  if (batch < 1 || batch > RV_MAX_BATCH) return rv_fail(RV_E_ARG, "batch must be in [1, %d]", RV_MAX_BATCH);
  if (k < 0 || k > RV_MAX_DRAFTS) return rv_fail(RV_E_ARG, "k must be in [0, %d]", RV_MAX_DRAFTS);
  if (k > 0 && !d_draft_ids) return rv_fail(RV_E_ARG, "draft ids are NULL");
  if (vocab < 1 || vocab > 64 * 2 * kChunk) return rv_fail(RV_E_ARG, "vocab must be in [1, %d]", 64 * 2 * kChunk);
  if (rv_status fs = rv_check_fusion(fusion); fs != RV_OK) return fs;
  if (fusion->rule == RV_RULE_SAMPLING) return rv_fail(RV_E_ARG, "the sampling rule is not available here");
  const int R1 = batch * (k + 1);
  const int nchunk = (vocab + kChunk - 1) / kChunk;
  const size_t part = (size_t)4 * R1 * nchunk * 4 * sizeof(float);
  const size_t rows = (size_t)R1 * sizeof(float);
  const size_t need = align256(part) + align256(3 * rows) + align256(2 * rows) + align256(rows) +
                      align256((size_t)batch * (k + 2) * sizeof(float));
  if ((size_t)R1 * nchunk > kMaxChunkRows || need > kScratchBytes)
    return rv_fail(RV_E_CAPACITY, "batch*(k+1)*ceil(vocab/%d) = %zu exceeds %zu (scratch of %zu bytes)", kChunk,
                   (size_t)R1 * nchunk, kMaxChunkRows, kScratchBytes);
  void* base = nullptr;
  if (rv_status s = scratch_on_current_device(&base); s != RV_OK) return s;

  char* p = (char*)base;
  HeadArgs a{};
  a.part = (float*)p;
  p += align256(part);
  a.lse = (float*)p;
  p += align256(3 * rows);
  a.entropy = (float*)p;
  p += align256(2 * rows);
  a.argmax = (int*)p;
  p += align256(rows);
  a.margins = (float*)p;
  a.B = batch;
  a.k = k;
  a.V = vocab;
  a.R1 = R1;
  for (int b = 0; b < batch; ++b) a.kb[b] = (uint8_t)k;
  a.nchunk = nchunk;
  a.chunk = kChunk;
  a.alpha = fusion->alpha;
  a.rule = fusion->rule;
  a.eps = fusion->epsilon;
  a.delta = fusion->delta;
  a.ent_src = fusion->entropy_src;
  a.temp = fusion->temperature;
  a.logits = d_logits;
  a.drafts = d_draft_ids;
  a.accept_len = d_accept_len;
  a.next_id = d_next_id;
  // z, lp, ids, row_bad, seq_bad stay NULL: no kept rows, no history, draft
  // ids checked against the vocabulary
  hipError_t e = launch_head(a, (hipStream_t)stream);
  if (e != hipSuccess) return rv_fail(RV_E_HIP, "accept: %s", hipGetErrorString(e));
  return RV_OK;
}
