// C ABI of the tiled contrastive loss: argument validation, workspace layout,
// grid selection and launches on the caller's stream.  No allocation, no host
// synchronisation, no global mutable state.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "infcl.h"

namespace infcl {
int launch_fwd(const void* img, const void* txt, int64_t b, int64_t d, int dtype, const float* scale, float* loss,
               double* loss64, float* lse_r, float* lse_c, float* aux, hipStream_t stream, float* rowR, float* rowL,
               float* colR, float* colL, float* udiag, float* ref2, double* partial);
int launch_fwd_shard(const void* img, const void* txt, int64_t b, int64_t d, int dtype, int64_t r0, int64_t nrows,
                     const float* scale, float* colpair, hipStream_t stream, float* rowR, float* rowL, float* colR,
                     float* colL, float* udiag, float* ref2);
int launch_fwd_shard_finish(int64_t b, int64_t d, int dtype, int64_t r0, int64_t nrows, int64_t nparts,
                            const float* colpairs, const float* scale, float* lse_r, float* lse_c, float* aux,
                            double* loss_part, hipStream_t stream, const float* rowR, const float* rowL,
                            const float* udiag, double* partial);
void fwd1_grid(int64_t b, int64_t nrows, int* Pr, int* Pc);
void fwd2_grid(int64_t b, int64_t nrows, int64_t d, int* Pr, int* Pc);
bool fwd2_supported(int64_t d, int dtype);
int launch_bwd(const void* img, const void* txt, int64_t b, int64_t d, int dtype, int64_t r0, int64_t nrows,
               const float* scale, const float* lse_r, const float* lse_c, const float* aux, const float* dloss,
               void* dimg, void* dtxt, int gdt, float* dscale, double* dscale64, float* lse2, double* ds_part,
               float* g16, hipStream_t stream);
bool bwd_supported(int64_t d, int dtype);
}  // namespace infcl

namespace {

constexpr int64_t kMaxB = (int64_t)1 << 30;

// Widths: the interface takes 16-bit rows of any multiple of 8 features up to
// 1024 and fp32 rows of any multiple of 4 up to 512 (16-byte rows); the sweeps
// are built for multiples of 128 (16-bit) and 64 (fp32), and other widths run
// on zero-padded copies of the inputs in the workspace, the gradients going
// through padded buffers there too.  Zero features add nothing to any dot
// product, so every output is that of the unpadded problem; the padding's
// gradients are zero and are dropped.
int64_t kernel_width(int64_t d, int dtype) {
  const int64_t q = dtype == INFCL_F32 ? 64 : 128;
  return (d + q - 1) / q * q;
}
bool width_ok(int64_t d, int dtype) { return dtype == INFCL_F32 ? d % 4 == 0 && d <= 512 : d % 8 == 0 && d <= 1024; }
size_t elem_size(int dtype) { return dtype == INFCL_F32 ? 4 : 2; }

struct Layout {
  int64_t dk;  // the width the sweeps run at
  size_t rowR, rowL, colR, colL, udiag, ref2, fwd_part, lse2, bwd_part, g16, pad, gpad, total;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Workspace regions, sized for the sweeps that (b, d, dtype) launches: the
// partial pairs of the forward grid (resident rows: Pc row and Pr column
// partials per sample; streamed tiles: 4 Pc and Pr), the diagonal, the base-2
// diagonal references (resident rows only), the loss and dscale partials, the
// base-2 log-sum-exp vectors of the backward and fp16's G' scale.  A shard of
// nrows <= b rows needs no more: its grid has at most as many row groups and
// its row partials are nrows long.
Layout make_layout(int64_t b, int64_t d, int dtype) {
  Layout L;
  L.dk = kernel_width(d, dtype);
  int Pr = 0, Pc = 0;
  size_t nrow = 0, ncol = 0;
  const bool resident = infcl::fwd2_supported(L.dk, dtype);
  if (resident) {
    infcl::fwd2_grid(b, b, L.dk, &Pr, &Pc);
    nrow = (size_t)Pc;
  } else {
    infcl::fwd1_grid(b, b, &Pr, &Pc);
    nrow = (size_t)Pc * 4;
  }
  ncol = (size_t)Pr;
  size_t off = 0;
  const size_t fb = (size_t)b * sizeof(float);
  L.rowR = off; off = align256(off + nrow * fb);
  L.rowL = off; off = align256(off + nrow * fb);
  L.colR = off; off = align256(off + ncol * fb);
  L.colL = off; off = align256(off + ncol * fb);
  L.udiag = off; off = align256(off + fb);
  L.ref2 = off; off = align256(off + (resident ? fb : 0));
  L.fwd_part = off; off = align256(off + (size_t)((b + 255) / 256) * sizeof(double));
  L.lse2 = off; off = align256(off + 2 * fb);
  L.bwd_part = off; off = align256(off + (size_t)2 * ((b + 63) / 64) * sizeof(double));  // 64 or 128 rows per WG
  L.g16 = off; off = align256(off + (dtype == INFCL_F16 ? (size_t)(2 + 2 * ((b + 255) / 256)) * sizeof(float) : 0));
  L.pad = off; off = align256(off + (L.dk != d ? 2 * (size_t)b * (size_t)L.dk * elem_size(dtype) : 0));  // img, txt
  L.gpad = off; off = align256(off + (L.dk != d ? 2 * (size_t)b * (size_t)L.dk * sizeof(float) : 0));  // dimg, dtxt
  L.total = off;
  return L;
}

// Row copy between widths: rows of cin 16-byte chunks into rows of cout
// chunks, cut or zero-filled at the end.
__global__ void __launch_bounds__(256) copy_rows(const uint4* __restrict__ src, uint4* __restrict__ dst, int64_t rows,
                                                 int cin, int cout) {
  const int64_t n = rows * cout;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = i / cout;
    const int c = (int)(i - r * cout);
    dst[i] = c < cin ? src[r * cin + c] : make_uint4(0u, 0u, 0u, 0u);
  }
}

unsigned copy_grid(int64_t n) { return (unsigned)(n / 256 + 1 < 65536 ? n / 256 + 1 : 65536); }

// The inputs the sweeps read: img and txt as given, or, when d is not a width
// the sweeps are built for, their zero-padded copies in the workspace.
// Returns false on a launch failure.
bool stage_inputs(const void*& img, const void*& txt, int64_t b, int64_t d, int dtype, char* ws, const Layout& L,
                  hipStream_t stream) {
  if (L.dk == d) return true;
  const int cin = (int)(d * elem_size(dtype) / 16), cout = (int)(L.dk * elem_size(dtype) / 16);
  const int64_t n = b * cout;
  uint4* pi = (uint4*)(ws + L.pad);
  uint4* pt = pi + n;
  hipLaunchKernelGGL(copy_rows, dim3(copy_grid(n)), dim3(256), 0, stream, (const uint4*)img, pi, b, cin, cout);
  hipLaunchKernelGGL(copy_rows, dim3(copy_grid(n)), dim3(256), 0, stream, (const uint4*)txt, pt, b, cin, cout);
  if (hipGetLastError() != hipSuccess) return false;
  img = pi;
  txt = pt;
  return true;
}

// Gradient element type: 0 fp32, 1 the 16-bit input type; -1 for an unknown
// type, -2 for a known one that is neither (16-bit gradients of another type,
// or of fp32 inputs, are not built).
int grad_kind(int grad_dtype, int dtype) {
  if (grad_dtype != INFCL_BF16 && grad_dtype != INFCL_F32 && grad_dtype != INFCL_F16) return -1;
  if (grad_dtype == INFCL_F32) return 0;
  return grad_dtype == dtype ? 1 : -2;
}

// Where the sweeps write the gradients of `rows` own samples: the caller's
// dimg and dtxt, or padded buffers in the workspace that unstage_grads then
// copies, without the padding, into the caller's.  ges: gradient element size.
void grad_targets(void*& gi, void*& gt, int64_t b, int64_t d, size_t ges, char* ws, const Layout& L) {
  if (L.dk == d) return;
  gi = ws + L.gpad;
  gt = ws + L.gpad + (size_t)b * (size_t)L.dk * ges;
}
bool unstage_grads(void* dimg, void* dtxt, int64_t rows, int64_t b, int64_t d, size_t ges, char* ws,
                   const Layout& L, hipStream_t stream) {
  if (L.dk == d) return true;
  const int cin = (int)(L.dk * ges / 16), cout = (int)(d * ges / 16);
  const uint4* gi = (const uint4*)(ws + L.gpad);
  const uint4* gt = gi + b * cin;
  const int64_t n = rows * cout;
  hipLaunchKernelGGL(copy_rows, dim3(copy_grid(n)), dim3(256), 0, stream, gi, (uint4*)dimg, rows, cin, cout);
  hipLaunchKernelGGL(copy_rows, dim3(copy_grid(n)), dim3(256), 0, stream, gt, (uint4*)dtxt, rows, cin, cout);
  return hipGetLastError() == hipSuccess;
}


bool aligned(const void* p, size_t a) { return p != nullptr && ((uintptr_t)p % a) == 0; }

bool shape_ok(int64_t b, int64_t d, int dtype) {
  return b >= 1 && d >= 1 && (dtype == INFCL_BF16 || dtype == INFCL_F32 || dtype == INFCL_F16);
}

bool shape_supported(int64_t b, int64_t d, int dtype) {
  return b <= kMaxB && width_ok(d, dtype) && infcl::bwd_supported(kernel_width(d, dtype), dtype);
}

// A shard: own samples [r0, r0 + bs) of the batch, r0 a multiple of 32 (so
// that own row blocks line up with the 32-row swept tiles).
bool shard_ok(int64_t b, int64_t r0, int64_t bs) { return r0 >= 0 && r0 % 32 == 0 && bs >= 1 && r0 + bs <= b; }

constexpr int64_t kMaxParts = 1 << 16;  // shards whose column pairs one finish merges

// ---- fixed scratch of infcl_fwd_noalloc: its workspace, for callers that
// cannot allocate.  Each device holds its own copy for the life of the
// process.  In host code the array's name is not a device address: the
// address comes from hipGetSymbolAddress, once per device, with that device
// current, and only that address is handed to kernels.
constexpr size_t kScratchBytes = (size_t)32 << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) char scratch[kScratchBytes];
void* g_scratch_ptr[kMaxDevices] = {};
std::mutex g_scratch_mu;

// The current device's scratch address (nullptr on a HIP error).
void* scratch_address() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

infcl_status infcl_workspace_size(int64_t b, int64_t d, int dtype, size_t* bytes) {
  if (bytes == nullptr || !shape_ok(b, d, dtype)) return INFCL_ERR_INVALID;
  if (!shape_supported(b, d, dtype)) return INFCL_ERR_UNSUPPORTED;
  *bytes = make_layout(b, d, dtype).total;
  return INFCL_OK;
}

infcl_status infcl_fwd(const void* img, const void* txt, int64_t b, int64_t d, int dtype, const float* scale,
                       float* loss, double* loss64, float* lse_r, float* lse_c, float* aux, void* workspace,
                       size_t ws_bytes, void* stream) {
  if (!shape_ok(b, d, dtype)) return INFCL_ERR_INVALID;
  if (!aligned(img, 16) || !aligned(txt, 16) || !aligned(scale, 4) || !aligned(loss, 4) || !aligned(lse_r, 16) ||
      !aligned(lse_c, 16) || !aligned(aux, 16) || !aligned(workspace, 256))
    return INFCL_ERR_INVALID;
  if (loss64 != nullptr && ((uintptr_t)loss64 % 8) != 0) return INFCL_ERR_INVALID;
  if (!shape_supported(b, d, dtype)) return INFCL_ERR_UNSUPPORTED;
  const Layout L = make_layout(b, d, dtype);
  if (ws_bytes < L.total) return INFCL_ERR_WORKSPACE;
  char* ws = (char*)workspace;
  if (!stage_inputs(img, txt, b, d, dtype, ws, L, (hipStream_t)stream)) return INFCL_ERR_HIP;
  int rc = infcl::launch_fwd(img, txt, b, L.dk, dtype, scale, loss, loss64, lse_r, lse_c, aux, (hipStream_t)stream,
                             (float*)(ws + L.rowR), (float*)(ws + L.rowL), (float*)(ws + L.colR),
                             (float*)(ws + L.colL), (float*)(ws + L.udiag), (float*)(ws + L.ref2),
                             (double*)(ws + L.fwd_part));
  return rc == 0 ? INFCL_OK : INFCL_ERR_HIP;
}

infcl_status infcl_fwd_noalloc(const void* img, const void* txt, int64_t b, int64_t d, int dtype, const float* scale,
                               float* loss, double* loss64, float* lse_r, float* lse_c, float* aux, void* stream) {
  if (!shape_ok(b, d, dtype)) return INFCL_ERR_INVALID;
  if (!aligned(img, 16) || !aligned(txt, 16) || !aligned(scale, 4) || !aligned(loss, 4) || !aligned(lse_r, 16) ||
      !aligned(lse_c, 16) || !aligned(aux, 16))
    return INFCL_ERR_INVALID;
  if (loss64 != nullptr && ((uintptr_t)loss64 % 8) != 0) return INFCL_ERR_INVALID;
  if (!shape_supported(b, d, dtype)) return INFCL_ERR_UNSUPPORTED;
  const Layout L = make_layout(b, d, dtype);
  if (L.total > kScratchBytes) return INFCL_ERR_WORKSPACE;
  char* ws = (char*)scratch_address();
  if (ws == nullptr) return INFCL_ERR_HIP;
  if (!stage_inputs(img, txt, b, d, dtype, ws, L, (hipStream_t)stream)) return INFCL_ERR_HIP;
  int rc = infcl::launch_fwd(img, txt, b, L.dk, dtype, scale, loss, loss64, lse_r, lse_c, aux, (hipStream_t)stream,
                             (float*)(ws + L.rowR), (float*)(ws + L.rowL), (float*)(ws + L.colR),
                             (float*)(ws + L.colL), (float*)(ws + L.udiag), (float*)(ws + L.ref2),
                             (double*)(ws + L.fwd_part));
  return rc == 0 ? INFCL_OK : INFCL_ERR_HIP;
}

infcl_status infcl_bwd(const void* img, const void* txt, int64_t b, int64_t d, int dtype, const float* scale,
                       const float* lse_r, const float* lse_c, const float* aux, const float* dloss, void* dimg,
                       void* dtxt, int grad_dtype, float* dscale, void* workspace, size_t ws_bytes, void* stream) {
  const int gk = grad_kind(grad_dtype, dtype);
  if (!shape_ok(b, d, dtype) || gk == -1) return INFCL_ERR_INVALID;
  if (!aligned(img, 16) || !aligned(txt, 16) || !aligned(scale, 4) || !aligned(lse_r, 16) || !aligned(lse_c, 16) ||
      !aligned(aux, 16) || !aligned(dimg, 16) || !aligned(dtxt, 16) || !aligned(dscale, 4) ||
      !aligned(workspace, 256))
    return INFCL_ERR_INVALID;
  if (dloss != nullptr && ((uintptr_t)dloss % 4) != 0) return INFCL_ERR_INVALID;
  if (!shape_supported(b, d, dtype) || gk < 0) return INFCL_ERR_UNSUPPORTED;
  const Layout L = make_layout(b, d, dtype);
  if (ws_bytes < L.total) return INFCL_ERR_WORKSPACE;
  char* ws = (char*)workspace;
  if (!stage_inputs(img, txt, b, d, dtype, ws, L, (hipStream_t)stream)) return INFCL_ERR_HIP;
  const size_t ges = gk ? 2 : 4;
  void *gi = dimg, *gt = dtxt;
  grad_targets(gi, gt, b, d, ges, ws, L);
  int rc = infcl::launch_bwd(img, txt, b, L.dk, dtype, 0, b, scale, lse_r, lse_c, aux, dloss, gi, gt, gk, dscale,
                             nullptr, (float*)(ws + L.lse2), (double*)(ws + L.bwd_part), (float*)(ws + L.g16),
                             (hipStream_t)stream);
  if (rc == 2) return INFCL_ERR_UNSUPPORTED;
  if (rc == 0 && !unstage_grads(dimg, dtxt, b, b, d, ges, ws, L, (hipStream_t)stream)) rc = 1;
  return rc == 0 ? INFCL_OK : INFCL_ERR_HIP;
}

// ------------------------------------------------------------------ shards

infcl_status infcl_fwd_shard(const void* img, const void* txt, int64_t b, int64_t d, int dtype, int64_t r0,
                             int64_t bs, const float* scale, float* colpair, void* workspace, size_t ws_bytes,
                             void* stream) {
  if (!shape_ok(b, d, dtype) || !shard_ok(b, r0, bs)) return INFCL_ERR_INVALID;
  if (!aligned(img, 16) || !aligned(txt, 16) || !aligned(scale, 4) || !aligned(colpair, 16) ||
      !aligned(workspace, 256))
    return INFCL_ERR_INVALID;
  if (!shape_supported(b, d, dtype)) return INFCL_ERR_UNSUPPORTED;
  const Layout L = make_layout(b, d, dtype);
  if (ws_bytes < L.total) return INFCL_ERR_WORKSPACE;
  char* ws = (char*)workspace;
  if (!stage_inputs(img, txt, b, d, dtype, ws, L, (hipStream_t)stream)) return INFCL_ERR_HIP;
  int rc = infcl::launch_fwd_shard(img, txt, b, L.dk, dtype, r0, bs, scale, colpair, (hipStream_t)stream,
                                   (float*)(ws + L.rowR), (float*)(ws + L.rowL), (float*)(ws + L.colR),
                                   (float*)(ws + L.colL), (float*)(ws + L.udiag), (float*)(ws + L.ref2));
  return rc == 0 ? INFCL_OK : INFCL_ERR_HIP;
}

infcl_status infcl_fwd_shard_finish(int64_t b, int64_t d, int dtype, int64_t r0, int64_t bs, int64_t nparts,
                                    const float* colpairs, const float* scale, float* lse_r, float* lse_c,
                                    float* aux, double* loss_part, void* workspace, size_t ws_bytes, void* stream) {
  if (!shape_ok(b, d, dtype) || !shard_ok(b, r0, bs) || nparts < 1 || nparts > kMaxParts) return INFCL_ERR_INVALID;
  if (!aligned(colpairs, 4) || !aligned(scale, 4) || !aligned(lse_r, 4) || !aligned(lse_c, 4) || !aligned(aux, 4) ||
      !aligned(loss_part, 8) || !aligned(workspace, 256))
    return INFCL_ERR_INVALID;
  if (!shape_supported(b, d, dtype)) return INFCL_ERR_UNSUPPORTED;
  const Layout L = make_layout(b, d, dtype);
  if (ws_bytes < L.total) return INFCL_ERR_WORKSPACE;
  char* ws = (char*)workspace;
  int rc = infcl::launch_fwd_shard_finish(b, L.dk, dtype, r0, bs, nparts, colpairs, scale, lse_r, lse_c, aux, loss_part,
                                          (hipStream_t)stream, (const float*)(ws + L.rowR),
                                          (const float*)(ws + L.rowL), (const float*)(ws + L.udiag),
                                          (double*)(ws + L.fwd_part));
  return rc == 0 ? INFCL_OK : INFCL_ERR_HIP;
}

infcl_status infcl_bwd_shard(const void* img, const void* txt, int64_t b, int64_t d, int dtype, int64_t r0,
                             int64_t bs, const float* scale, const float* lse_r, const float* lse_c, const float* aux,
                             const float* dloss, void* dimg, void* dtxt, int grad_dtype, double* dscale_part,
                             void* workspace, size_t ws_bytes, void* stream) {
  const int gk = grad_kind(grad_dtype, dtype);
  if (!shape_ok(b, d, dtype) || !shard_ok(b, r0, bs) || gk == -1) return INFCL_ERR_INVALID;
  if (!aligned(img, 16) || !aligned(txt, 16) || !aligned(scale, 4) || !aligned(lse_r, 16) || !aligned(lse_c, 16) ||
      !aligned(aux, 16) || !aligned(dimg, 16) || !aligned(dtxt, 16) || !aligned(dscale_part, 8) ||
      !aligned(workspace, 256))
    return INFCL_ERR_INVALID;
  if (dloss != nullptr && ((uintptr_t)dloss % 4) != 0) return INFCL_ERR_INVALID;
  if (!shape_supported(b, d, dtype) || gk < 0) return INFCL_ERR_UNSUPPORTED;
  const Layout L = make_layout(b, d, dtype);
  if (ws_bytes < L.total) return INFCL_ERR_WORKSPACE;
  char* ws = (char*)workspace;
  if (!stage_inputs(img, txt, b, d, dtype, ws, L, (hipStream_t)stream)) return INFCL_ERR_HIP;
  const size_t ges = gk ? 2 : 4;
  void *gi = dimg, *gt = dtxt;
  grad_targets(gi, gt, b, d, ges, ws, L);
  int rc = infcl::launch_bwd(img, txt, b, L.dk, dtype, r0, bs, scale, lse_r, lse_c, aux, dloss, gi, gt, gk, nullptr,
                             dscale_part, (float*)(ws + L.lse2), (double*)(ws + L.bwd_part), (float*)(ws + L.g16),
                             (hipStream_t)stream);
  if (rc == 2) return INFCL_ERR_UNSUPPORTED;
  if (rc == 0 && !unstage_grads(dimg, dtxt, bs, b, d, ges, ws, L, (hipStream_t)stream)) rc = 1;
  return rc == 0 ? INFCL_OK : INFCL_ERR_HIP;
}

const char* infcl_status_str(int status) {
  switch (status) {
    case INFCL_OK: return "ok";
    case INFCL_ERR_INVALID: return "invalid argument (null or misaligned pointer, b < 1, d < 1 or unknown dtype)";
    case INFCL_ERR_UNSUPPORTED:
      return "unsupported shape (bf16, f16: d a multiple of 8 up to 1024; f32: d a multiple of 4 up to 512; "
             "b <= 2^30) or gradient type (f32, or the inputs' 16-bit type)";
    case INFCL_ERR_WORKSPACE: return "workspace smaller than infcl_workspace_size()";
    case INFCL_ERR_HIP: return "HIP kernel launch failed";
    default: return "unknown status";
  }
}

}  // extern "C"
