// C entry points: argument checks, workspace sizing and launches.  No
// allocation and no host synchronisation.  The only global state is that of
// the allocation-free acceptance: its static device scratch array and the
// per-device cache of that array's address.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "treeverify.h"
#include "tv_plan.h"

static_assert(TV_MAX_NODES == tv::kMaxNodes, "node limit mismatch");
static_assert(TV_MAX_DRAFT_DEPTH == tv::kMaxDraftDepth, "draft depth limit");

namespace tv {
hipError_t launch_attention(const void* q, const void* kc, const void* vc, const void* kt,
                            const void* vt, const int32_t* parent, const int32_t* kv_len,
                            void* out, int B, int N, int Hq, int Hkv, int D, int Lmax,
                            float scale, void* ws, const AttnPlan& p, hipStream_t st,
                            const int32_t* block_table, int block_shift, int max_blocks,
                            int num_blocks, int cgroup);
hipError_t launch_commit(const void* kt, const void* vt, const int32_t* path,
                         const int32_t* accept_len, void* kc, void* vc, int32_t* kv_len,
                         const int32_t* block_table, int shift, int max_blocks, int num_blocks,
                         int B, int N, int Hkv, int D, int cap, int Dmax, hipStream_t st);
hipError_t launch_accept(const void* logits, int f32, const int32_t* draft, const int32_t* parent,
                         int B, int N, int V, int Dmax, int32_t* accept_len, int32_t* path,
                         int32_t* tgt_out, void* ws, hipStream_t st);
hipError_t launch_topw(const void* logits, int f32, int B, int Nd, int V, int W, int32_t* tok,
                       float* logp, void* ws, hipStream_t st);
hipError_t launch_sample(const void* logits, int f32, const int32_t* draft,
                         const int32_t* parent, const float* u, unsigned long long seed,
                         float temperature, int B, int N, int V, int Dmax, int32_t* accept_len,
                         int32_t* path, int32_t* corr, void* ws, hipStream_t st);
hipError_t launch_build_tree(const int32_t* tok, const float* logp, const int32_t* root_tok, int B,
                             int Nd, int W, int budget, int32_t* parent, int32_t* token,
                             int32_t* depth, float* score, int32_t* n_nodes, hipStream_t st);
}  // namespace tv

static_assert(TV_MAX_WIDTH == tv::kTopwMax, "width limit mismatch");

static bool misaligned(const void* p) { return ((uintptr_t)p & 15u) != 0; }

static int check_attention_sizes(int B, int N, int Hq, int Hkv, int D, int Lmax) {
  if (B < 1 || N < 1 || Hq < 1 || Hkv < 1 || Lmax < 0) return TV_ERR_SHAPE;
  if (Hq % Hkv != 0) return TV_ERR_SHAPE;
  if (D != 64 && D != 128) return TV_ERR_UNSUPPORTED;
  if (N > TV_MAX_NODES) return TV_ERR_UNSUPPORTED;
  // element offsets are formed in 64-bit, but row indices stay in int32
  if ((long long)B * N * Hq > (1ll << 31) || (long long)B * Lmax > (1ll << 31)) return TV_ERR_UNSUPPORTED;
  return TV_OK;
}

// log2 of a valid block size (a power of two in [32, 2^20]), else -1
static int block_shift(int block_size) {
  if (block_size < 32 || block_size > (1 << 20) || (block_size & (block_size - 1))) return -1;
  int s = 0;
  while ((1 << s) < block_size) ++s;
  return s;
}

// Tree K/V: both given, or both NULL for the tree-tail layout (node i at
// cache row kv_len + i), which needs room for the N tree rows in the cache.
static int check_tree(const void* kt, const void* vt, int N, int Lmax) {
  if (!kt != !vt) return TV_ERR_NULL;
  if (!kt && Lmax < N) return TV_ERR_SHAPE;
  if (misaligned(kt) || misaligned(vt)) return TV_ERR_ALIGN;
  return TV_OK;
}

// The training-mask attention runs as B*A chain trees of S nodes, block k of
// example b reading example b's context with kv_len = anchors[b, k].
static int check_block_causal(int B, int A, int S, int Hq, int Hkv, int D, int L) {
  if (A < 1 || S < 1 || B < 1) return TV_ERR_SHAPE;
  if ((long long)B * A > (1ll << 24)) return TV_ERR_UNSUPPORTED;
  return check_attention_sizes(B * A, S, Hq, Hkv, D, L);
}

static int check_accept_sizes(int B, int N, int V, int Dmax) {
  if (B < 1 || N < 1 || V < 1 || Dmax < 1) return TV_ERR_SHAPE;
  if (N > TV_MAX_NODES) return TV_ERR_UNSUPPORTED;
  if ((long long)B * N > (1ll << 24)) return TV_ERR_UNSUPPORTED;
  return TV_OK;
}

static int check_draft_sizes(int B, int Nd, int W) {
  if (B < 1 || Nd < 1 || W < 1) return TV_ERR_SHAPE;
  if (W > TV_MAX_WIDTH || Nd > TV_MAX_DRAFT_DEPTH) return TV_ERR_UNSUPPORTED;
  if ((long long)B * Nd > (1ll << 24)) return TV_ERR_UNSUPPORTED;
  return TV_OK;
}

extern "C" {

const char* tv_status_string(int status) {
  switch (status) {
    case TV_OK: return "TV_OK";
    case TV_ERR_NULL: return "TV_ERR_NULL: a required pointer is NULL";
    case TV_ERR_SHAPE: return "TV_ERR_SHAPE: invalid or inconsistent sizes";
    case TV_ERR_DTYPE: return "TV_ERR_DTYPE: unknown logits dtype";
    case TV_ERR_UNSUPPORTED: return "TV_ERR_UNSUPPORTED: shape outside the supported range";
    case TV_ERR_WORKSPACE: return "TV_ERR_WORKSPACE: workspace missing or too small";
    case TV_ERR_LAUNCH: return "TV_ERR_LAUNCH: the HIP runtime rejected a launch";
    case TV_ERR_ALIGN: return "TV_ERR_ALIGN: tensor pointer not 16-byte aligned";
    case TV_ERR_SCRATCH:
      return "TV_ERR_SCRATCH: sizes need more than the allocation-free entry point's static "
             "scratch (TV_ACCEPT_SCRATCH_BYTES)";
    default: return "unknown treeverify status";
  }
}

int tv_version(void) { return 2; }

size_t tv_tree_verify_attention_workspace(int B, int N, int Hq, int Hkv, int D, int Lmax) {
  if (check_attention_sizes(B, N, Hq, Hkv, D, Lmax) != TV_OK) return 0;
  const tv::AttnPlan p = tv::attn_plan(B, N, Hq, Hkv, D, Lmax);
  return p.ws_bytes > 0 ? p.ws_bytes : 256;
}

int tv_tree_verify_attention(const void* q, const void* k_cache, const void* v_cache,
                             const void* k_tree, const void* v_tree, const int32_t* parent,
                             const int32_t* kv_len, void* out, int B, int N, int Hq, int Hkv,
                             int D, int Lmax, float scale, void* workspace,
                             size_t workspace_bytes, hipStream_t stream) {
  int rc = check_attention_sizes(B, N, Hq, Hkv, D, Lmax);
  if (rc != TV_OK) return rc;
  if (!q || !parent || !out) return TV_ERR_NULL;
  if ((rc = check_tree(k_tree, v_tree, N, Lmax)) != TV_OK) return rc;
  if (Lmax > 0 && (!k_cache || !v_cache)) return TV_ERR_NULL;
  if (misaligned(q) || misaligned(out) ||
      (Lmax > 0 && (misaligned(k_cache) || misaligned(v_cache))))
    return TV_ERR_ALIGN;
  const tv::AttnPlan p = tv::attn_plan(B, N, Hq, Hkv, D, Lmax);
  if (p.ws_bytes > 0 && (!workspace || workspace_bytes < p.ws_bytes)) return TV_ERR_WORKSPACE;
  if (misaligned(workspace)) return TV_ERR_ALIGN;
  if (!(scale > 0.f)) scale = 1.0f / sqrtf((float)D);
  hipError_t e = tv::launch_attention(q, k_cache, v_cache, k_tree, v_tree, parent, kv_len, out,
                                      B, N, Hq, Hkv, D, Lmax, scale, workspace, p, stream,
                                      nullptr, 0, 0, 0, 1);
  return e == hipSuccess ? TV_OK : TV_ERR_LAUNCH;
}

size_t tv_block_causal_attention_workspace(int B, int A, int S, int Hq, int Hkv, int D,
                                          int L) {
  if (check_block_causal(B, A, S, Hq, Hkv, D, L) != TV_OK) return 0;
  const tv::AttnPlan p = tv::attn_plan(B * A, S, Hq, Hkv, D, L);
  return p.ws_bytes > 0 ? p.ws_bytes : 256;
}

int tv_block_causal_attention(const void* q, const void* k_ctx, const void* v_ctx,
                              const void* k_blk, const void* v_blk, const int32_t* anchors,
                              void* out, int B, int A, int S, int Hq, int Hkv, int D, int L,
                              float scale, void* workspace, size_t workspace_bytes,
                              hipStream_t stream) {
  int rc = check_block_causal(B, A, S, Hq, Hkv, D, L);
  if (rc != TV_OK) return rc;
  if (!q || !k_blk || !v_blk || !anchors || !out) return TV_ERR_NULL;
  if (L > 0 && (!k_ctx || !v_ctx)) return TV_ERR_NULL;
  if (misaligned(q) || misaligned(k_blk) || misaligned(v_blk) || misaligned(out) ||
      (L > 0 && (misaligned(k_ctx) || misaligned(v_ctx))))
    return TV_ERR_ALIGN;
  const tv::AttnPlan p = tv::attn_plan(B * A, S, Hq, Hkv, D, L);
  if (p.ws_bytes > 0 && (!workspace || workspace_bytes < p.ws_bytes)) return TV_ERR_WORKSPACE;
  if (misaligned(workspace)) return TV_ERR_ALIGN;
  if (!(scale > 0.f)) scale = 1.0f / sqrtf((float)D);
  hipError_t e = tv::launch_attention(q, k_ctx, v_ctx, k_blk, v_blk, nullptr, anchors, out,
                                      B * A, S, Hq, Hkv, D, L, scale, workspace, p, stream,
                                      nullptr, 0, 0, 0, A);
  return e == hipSuccess ? TV_OK : TV_ERR_LAUNCH;
}

int tv_tree_verify_attention_paged(const void* q, const void* k_pool, const void* v_pool,
                                   const int32_t* block_table, int block_size, int max_blocks,
                                   int num_blocks, const void* k_tree, const void* v_tree,
                                   const int32_t* parent, const int32_t* kv_len, void* out,
                                   int B, int N, int Hq, int Hkv, int D, float scale,
                                   void* workspace, size_t workspace_bytes,
                                   hipStream_t stream) {
  const int shift = block_shift(block_size);
  if (shift < 0 || max_blocks < 0 || num_blocks < 0) return TV_ERR_SHAPE;
  if ((long long)max_blocks * block_size > (1ll << 30)) return TV_ERR_UNSUPPORTED;
  const int Lmax = max_blocks * block_size;
  int rc = check_attention_sizes(B, N, Hq, Hkv, D, Lmax);
  if (rc != TV_OK) return rc;
  if (!q || !parent || !out) return TV_ERR_NULL;
  if ((rc = check_tree(k_tree, v_tree, N, Lmax)) != TV_OK) return rc;
  if (Lmax > 0 && (!k_pool || !v_pool || !block_table || num_blocks < 1)) return TV_ERR_NULL;
  if (misaligned(q) || misaligned(out) ||
      (Lmax > 0 && (misaligned(k_pool) || misaligned(v_pool))))
    return TV_ERR_ALIGN;
  const tv::AttnPlan p = tv::attn_plan(B, N, Hq, Hkv, D, Lmax);
  if (p.ws_bytes > 0 && (!workspace || workspace_bytes < p.ws_bytes)) return TV_ERR_WORKSPACE;
  if (misaligned(workspace)) return TV_ERR_ALIGN;
  if (!(scale > 0.f)) scale = 1.0f / sqrtf((float)D);
  hipError_t e = tv::launch_attention(q, k_pool, v_pool, k_tree, v_tree, parent, kv_len, out, B,
                                      N, Hq, Hkv, D, Lmax, scale, workspace, p, stream,
                                      Lmax > 0 ? block_table : nullptr, shift, max_blocks,
                                      num_blocks, 1);
  return e == hipSuccess ? TV_OK : TV_ERR_LAUNCH;
}

static int check_commit(const void* kt, const void* vt, const int32_t* path,
                        const int32_t* accept_len, const void* kc, const void* vc,
                        const int32_t* kv_len, int B, int N, int Hkv, int D, int Dmax, int cap) {
  if (B < 1 || N < 1 || Hkv < 1 || Dmax < 1 || cap < 1) return TV_ERR_SHAPE;
  if (D != 64 && D != 128) return TV_ERR_UNSUPPORTED;
  if (N > TV_MAX_NODES) return TV_ERR_UNSUPPORTED;
  if (!path || !accept_len || !kc || !vc || !kv_len) return TV_ERR_NULL;
  const int rc = check_tree(kt, vt, N, cap);
  if (rc != TV_OK) return rc;
  if (misaligned(kc) || misaligned(vc)) return TV_ERR_ALIGN;
  return TV_OK;
}

int tv_commit_path(const void* k_tree, const void* v_tree, const int32_t* path,
                   const int32_t* accept_len, void* k_cache, void* v_cache, int32_t* kv_len,
                   int B, int N, int Hkv, int D, int Lmax, int Dmax, hipStream_t stream) {
  int rc = check_commit(k_tree, v_tree, path, accept_len, k_cache, v_cache, kv_len, B, N, Hkv,
                        D, Dmax, Lmax);
  if (rc != TV_OK) return rc;
  if ((long long)B * Lmax > (1ll << 31)) return TV_ERR_UNSUPPORTED;
  hipError_t e = tv::launch_commit(k_tree, v_tree, path, accept_len, k_cache, v_cache, kv_len,
                                   nullptr, 0, 0, 0, B, N, Hkv, D, Lmax, Dmax, stream);
  return e == hipSuccess ? TV_OK : TV_ERR_LAUNCH;
}

int tv_commit_path_paged(const void* k_tree, const void* v_tree, const int32_t* path,
                         const int32_t* accept_len, void* k_pool, void* v_pool,
                         const int32_t* block_table, int block_size, int max_blocks,
                         int num_blocks, int32_t* kv_len, int B, int N, int Hkv, int D, int Dmax,
                         hipStream_t stream) {
  const int shift = block_shift(block_size);
  if (shift < 0 || max_blocks < 1 || num_blocks < 1) return TV_ERR_SHAPE;
  if ((long long)max_blocks * block_size > (1ll << 30)) return TV_ERR_UNSUPPORTED;
  int rc = check_commit(k_tree, v_tree, path, accept_len, k_pool, v_pool, kv_len, B, N, Hkv, D,
                        Dmax, max_blocks * block_size);
  if (rc != TV_OK) return rc;
  if (!block_table) return TV_ERR_NULL;
  hipError_t e = tv::launch_commit(k_tree, v_tree, path, accept_len, k_pool, v_pool, kv_len,
                                   block_table, shift, max_blocks, num_blocks, B, N, Hkv, D,
                                   max_blocks * block_size, Dmax, stream);
  return e == hipSuccess ? TV_OK : TV_ERR_LAUNCH;
}

size_t tv_tree_accept_workspace(int B, int N, int V) {
  if (check_accept_sizes(B, N, V, 1) != TV_OK) return 0;
  return tv::accept_ws_bytes(B, N);
}

int tv_tree_accept(const void* logits, int logits_dtype, const int32_t* draft_tok,
                   const int32_t* parent, int B, int N, int V, int Dmax, int32_t* accept_len,
                   int32_t* path, int32_t* tgt_argmax, void* workspace, size_t workspace_bytes,
                   hipStream_t stream) {
  int rc = check_accept_sizes(B, N, V, Dmax);
  if (rc != TV_OK) return rc;
  if (logits_dtype != TV_BF16 && logits_dtype != TV_F32) return TV_ERR_DTYPE;
  if (!logits || !draft_tok || !parent || !accept_len || !path) return TV_ERR_NULL;
  if (!workspace || workspace_bytes < tv::accept_ws_bytes(B, N)) return TV_ERR_WORKSPACE;
  if (misaligned(workspace)) return TV_ERR_ALIGN;
  hipError_t e = tv::launch_accept(logits, logits_dtype == TV_F32, draft_tok, parent, B, N, V,
                                   Dmax, accept_len, path, tgt_argmax, workspace, stream);
  return e == hipSuccess ? TV_OK : TV_ERR_LAUNCH;
}

// ---------------------------------------------------------------- static scratch
// The split keys of tv_tree_accept_noalloc live in this device array: every
// GPU the library runs on holds its own copy, from the code object's load
// until the process ends.  In host code the name is only a stand-in for the
// symbol, never a device address: the address of the current device's copy
// comes from hipGetSymbolAddress, once per device, and only that address is
// passed to kernels.
static __device__ __align__(256) unsigned char scratch[TV_ACCEPT_SCRATCH_BYTES];

constexpr int kScratchDevices = 64;
static std::atomic<void*> g_scratch_addr[kScratchDevices];

// Address of `stream`'s device's copy of the scratch array (the device is
// made current for the lookup and restored afterwards).
static int scratch_address(hipStream_t stream, void** out) {
  int dev = -1;
  if (stream) {
    hipDevice_t d;
    if (hipStreamGetDevice(stream, &d) != hipSuccess) return TV_ERR_LAUNCH;
    dev = (int)d;
  } else if (hipGetDevice(&dev) != hipSuccess) {
    return TV_ERR_LAUNCH;
  }
  if (dev < 0 || dev >= kScratchDevices) return TV_ERR_UNSUPPORTED;
  void* p = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (!p) {
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return TV_ERR_LAUNCH;
    if (cur != dev && hipSetDevice(dev) != hipSuccess) return TV_ERR_LAUNCH;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev && hipSetDevice(cur) != hipSuccess) return TV_ERR_LAUNCH;
    if (e != hipSuccess || !p) return TV_ERR_LAUNCH;
    g_scratch_addr[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return TV_OK;
}

int tv_tree_accept_noalloc(const void* logits, int logits_dtype, const int32_t* draft_tok,
                           const int32_t* parent, int B, int N, int V, int Dmax,
                           int32_t* accept_len, int32_t* path, int32_t* tgt_argmax,
                           hipStream_t stream) {
  int rc = check_accept_sizes(B, N, V, Dmax);
  if (rc != TV_OK) return rc;
  if (logits_dtype != TV_BF16 && logits_dtype != TV_F32) return TV_ERR_DTYPE;
  if (!logits || !draft_tok || !parent || !accept_len || !path) return TV_ERR_NULL;
  if (tv::accept_ws_bytes(B, N) > (size_t)TV_ACCEPT_SCRATCH_BYTES) return TV_ERR_SCRATCH;
  void* ws = nullptr;
  if ((rc = scratch_address(stream, &ws)) != TV_OK) return rc;
  // every split key is written by the scan before the finish reads it:
  // nothing in the scratch has to start at zero
  hipError_t e = tv::launch_accept(logits, logits_dtype == TV_F32, draft_tok, parent, B, N, V,
                                   Dmax, accept_len, path, tgt_argmax, ws, stream);
  return e == hipSuccess ? TV_OK : TV_ERR_LAUNCH;
}

static int check_sampled_sizes(int B, int N, int V, int Dmax) {
  const int rc = check_accept_sizes(B, N, V, Dmax);
  if (rc != TV_OK) return rc;
  if ((long long)V > tv::kMaxSampledVocab) return TV_ERR_UNSUPPORTED;
  return TV_OK;
}

size_t tv_tree_accept_sampled_workspace(int B, int N, int V) {
  if (check_sampled_sizes(B, N, V, 1) != TV_OK) return 0;
  return tv::sample_plan(B, N, V).ws_bytes;
}

int tv_tree_accept_sampled(const void* logits, int logits_dtype, const int32_t* draft_tok,
                           const int32_t* parent, const float* u_accept, unsigned long long seed,
                           float temperature, int B, int N, int V, int Dmax, int32_t* accept_len,
                           int32_t* path, int32_t* correction, void* workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  int rc = check_sampled_sizes(B, N, V, Dmax);
  if (rc != TV_OK) return rc;
  if (!(temperature > 0.f) || !(temperature < INFINITY)) return TV_ERR_SHAPE;
  if (logits_dtype != TV_BF16 && logits_dtype != TV_F32) return TV_ERR_DTYPE;
  if (!logits || !draft_tok || !parent || !u_accept || !accept_len || !path || !correction)
    return TV_ERR_NULL;
  const tv::SamplePlan p = tv::sample_plan(B, N, V);
  if (!workspace || workspace_bytes < p.ws_bytes) return TV_ERR_WORKSPACE;
  if (misaligned(workspace)) return TV_ERR_ALIGN;
  hipError_t e = tv::launch_sample(logits, logits_dtype == TV_F32, draft_tok, parent, u_accept,
                                   seed, temperature, B, N, V, Dmax, accept_len, path,
                                   correction, workspace, stream);
  return e == hipSuccess ? TV_OK : TV_ERR_LAUNCH;
}

size_t tv_draft_topw_workspace(int B, int Nd, int V) {
  if (check_draft_sizes(B, Nd, 1) != TV_OK || V < 1) return 0;
  return tv::topw_ws_bytes(B, Nd);
}

int tv_draft_topw(const void* logits, int logits_dtype, int B, int Nd, int V, int W,
                  int32_t* tok, float* logp, void* workspace, size_t workspace_bytes,
                  hipStream_t stream) {
  int rc = check_draft_sizes(B, Nd, W);
  if (rc != TV_OK) return rc;
  if (V < 1 || W > V) return TV_ERR_SHAPE;
  if (logits_dtype != TV_BF16 && logits_dtype != TV_F32) return TV_ERR_DTYPE;
  if (!logits || !tok || !logp) return TV_ERR_NULL;
  if (!workspace || workspace_bytes < tv::topw_ws_bytes(B, Nd)) return TV_ERR_WORKSPACE;
  if (misaligned(workspace)) return TV_ERR_ALIGN;
  hipError_t e = tv::launch_topw(logits, logits_dtype == TV_F32, B, Nd, V, W, tok, logp,
                                 workspace, stream);
  return e == hipSuccess ? TV_OK : TV_ERR_LAUNCH;
}

int tv_build_tree(const int32_t* tok, const float* logp, const int32_t* root_tok, int B,
                  int Nd, int W, int budget, int32_t* parent, int32_t* token, int32_t* depth,
                  float* score, int32_t* n_nodes, hipStream_t stream) {
  int rc = check_draft_sizes(B, Nd, W);
  if (rc != TV_OK) return rc;
  if (budget < 1) return TV_ERR_SHAPE;
  if (budget > TV_MAX_NODES) return TV_ERR_UNSUPPORTED;
  if (!tok || !logp || !parent || !token || !depth || !n_nodes) return TV_ERR_NULL;
  hipError_t e = tv::launch_build_tree(tok, logp, root_tok, B, Nd, W, budget, parent, token,
                                       depth, score, n_nodes, stream);
  return e == hipSuccess ? TV_OK : TV_ERR_LAUNCH;
}

}  // extern "C"
