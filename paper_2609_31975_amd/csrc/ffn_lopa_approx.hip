// LoPA approximation of a gate matrix (include/ffn_lopa_approx.h): alternating M steps
// (a kernel) and truncated-SVD steps (rocBLAS Gram matrix and products, rocSOLVER
// symmetric eigensolver), all in fp64.
//
// Layouts: W, W - M and the residual are row-major [H][D]; rocBLAS sees such a matrix as
// its column-major transpose (D x H, leading dimension D).  With Ac = (W - M)^T in that
// view, the Gram matrix G = (W - M)^T (W - M) = Ac Ac^T (D x D, symmetric) comes from
// SYRK; its eigenvectors (columns of G after the eigensolver, eigenvalues ascending) for
// the r largest eigenvalues are the right singular vectors: V row k = eigenvector
// D - 1 - k.  U = (W - M) V^T, as U^T (r x H column-major = U row-major) = V Ac, and the
// residual W - U V = W - (V^T U^T)^T, as Rc = Wc - Vc Ut with Vc = V^T (D x r).
#include <math.h>
#include <stdint.h>

#include <rocblas/rocblas.h>
#include <rocsolver/rocsolver.h>

#include "ffn_lopa_approx.h"
#include "ffn_sparse.h"

namespace {

constexpr int kThreads = 256;

size_t round_up(size_t v) { return (v + 255) / 256 * 256; }

struct Ws {
  double* R;       // [H][D]: W - M, then the residual W - U V
  double* G;       // [D][D]: Gram matrix, then its eigenvectors
  double* eig;     // [D]
  double* E;       // [D] eigensolver scratch
  double* Ut;      // [H][r]: U
  double* V;       // [r][D]
  double* part;    // [H]: per-row error terms
  double* total;   // [1]
  int32_t* idx[2];  // [H] M's column, current and next
  int8_t* sgn[2];   // [H] M's value
  int* flags;       // [0] M changed, [1] eigensolver info
};

size_t layout(int H, int D, int r, void* base, Ws* w) {
  size_t off = 0;
  char* b = static_cast<char*>(base);
  auto take = [&](size_t bytes) {
    char* p = b ? b + off : nullptr;
    off += round_up(bytes);
    return p;
  };
  Ws o{};
  o.R = reinterpret_cast<double*>(take(8 * (size_t)H * D));
  o.G = reinterpret_cast<double*>(take(8 * (size_t)D * D));
  o.eig = reinterpret_cast<double*>(take(8 * (size_t)D));
  o.E = reinterpret_cast<double*>(take(8 * (size_t)D));
  o.Ut = reinterpret_cast<double*>(take(8 * (size_t)H * r));
  o.V = reinterpret_cast<double*>(take(8 * (size_t)r * D));
  o.part = reinterpret_cast<double*>(take(8 * (size_t)H));
  o.total = reinterpret_cast<double*>(take(8));
  for (int i = 0; i < 2; ++i) {
    o.idx[i] = reinterpret_cast<int32_t*>(take(4 * (size_t)H));
    o.sgn[i] = reinterpret_cast<int8_t*>(take((size_t)H));
  }
  o.flags = reinterpret_cast<int*>(take(16));
  if (w) *w = o;
  return off;
}

// R = W - M (M given, or none) in fp64
__global__ void k_w_minus_m(const float* __restrict__ w, const int32_t* __restrict__ idx,
                            const int8_t* __restrict__ sgn, double* __restrict__ R, int H, int D) {
  const size_t n = (size_t)H * D;
  for (size_t e = blockIdx.x * (size_t)kThreads + threadIdx.x; e < n; e += (size_t)gridDim.x * kThreads) {
    const int i = (int)(e / (size_t)D), j = (int)(e - (size_t)i * D);
    double v = (double)w[e];
    if (idx && idx[i] == j) v -= (double)sgn[i];
    R[e] = v;
  }
}

// M step on the residual R: one workgroup per row.  Writes the new column and sign, the
// row's error for the old M (if any) and for the new one, and flags a change.
__global__ void k_m_step(const double* __restrict__ R, int D, const int32_t* __restrict__ old_idx,
                         const int8_t* __restrict__ old_sgn, int32_t* __restrict__ new_idx,
                         int8_t* __restrict__ new_sgn, double* __restrict__ part, int* __restrict__ changed) {
  __shared__ double s_m[kThreads], s_q[kThreads];
  __shared__ int s_j[kThreads];
  const int i = blockIdx.x;
  const double* row = R + (size_t)i * D;
  double best = -1.0, q = 0.0;
  int bj = 0;
  for (int j = threadIdx.x; j < D; j += kThreads) {
    const double v = row[j];
    q += v * v;
    if (fabs(v) > best) {  // strictly greater: the lowest column of this thread's share wins
      best = fabs(v);
      bj = j;
    }
  }
  s_m[threadIdx.x] = best;
  s_j[threadIdx.x] = bj;
  s_q[threadIdx.x] = q;
  __syncthreads();
  for (int h = kThreads / 2; h > 0; h >>= 1) {
    if ((int)threadIdx.x < h) {
      const double a = s_m[threadIdx.x], b = s_m[threadIdx.x + h];
      const int ja = s_j[threadIdx.x], jb = s_j[threadIdx.x + h];
      if (b > a || (b == a && jb < ja)) {
        s_m[threadIdx.x] = b;
        s_j[threadIdx.x] = jb;
      }
      s_q[threadIdx.x] += s_q[threadIdx.x + h];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const int j = s_j[0];
    const double v = row[j];
    const int8_t s = v >= 0.0 ? 1 : -1;
    new_idx[i] = j;
    new_sgn[i] = s;
    // ||R_i - s e_j||^2 = ||R_i||^2 - 2 s R_ij + 1, for the new M
    part[i] = s_q[0] - 2.0 * (double)s * v + 1.0;
    if (old_idx && (old_idx[i] != j || old_sgn[i] != s)) changed[0] = 1;
  }
}

__global__ void k_sum(const double* __restrict__ part, int n, double* __restrict__ out) {
  __shared__ double s[kThreads];
  double a = 0.0;
  for (int i = threadIdx.x; i < n; i += kThreads) a += part[i];
  s[threadIdx.x] = a;
  __syncthreads();
  for (int h = kThreads / 2; h > 0; h >>= 1) {
    if ((int)threadIdx.x < h) s[threadIdx.x] += s[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = s[0];
}

// V[k][:] = eigenvector D-1-k (column D-1-k of G, contiguous)
__global__ void k_top_vectors(const double* __restrict__ G, int D, int r, double* __restrict__ V) {
  const size_t n = (size_t)r * D;
  for (size_t e = blockIdx.x * (size_t)kThreads + threadIdx.x; e < n; e += (size_t)gridDim.x * kThreads) {
    const int k = (int)(e / (size_t)D), j = (int)(e - (size_t)k * D);
    V[e] = G[(size_t)(D - 1 - k) * D + j];
  }
}

__global__ void k_to_f32(const double* __restrict__ a, float* __restrict__ b, size_t n) {
  for (size_t e = blockIdx.x * (size_t)kThreads + threadIdx.x; e < n; e += (size_t)gridDim.x * kThreads)
    b[e] = (float)a[e];
}

__global__ void k_copy_m(const int32_t* __restrict__ si, const int8_t* __restrict__ ss, int32_t* __restrict__ di,
                         int8_t* __restrict__ ds, int H) {
  for (int i = blockIdx.x * kThreads + threadIdx.x; i < H; i += gridDim.x * kThreads) {
    di[i] = si[i];
    ds[i] = ss[i];
  }
}

int grid_for(size_t n) {
  const size_t g = (n + kThreads - 1) / kThreads;
  return (int)(g < 8192 ? (g > 0 ? g : 1) : 8192);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool shape_ok(int H, int D, int r) {
  return H >= 1 && D >= 1 && r >= 1 && r <= (H < D ? H : D) && (int64_t)H * D < (int64_t(1) << 31);
}

struct Handle {
  rocblas_handle h = nullptr;
  ~Handle() {
    if (h) rocblas_destroy_handle(h);
  }
};

}  // namespace

extern "C" {

size_t ffn_lopa_approx_workspace_bytes(int H, int D, int r) {
  if (!shape_ok(H, D, r)) return 0;
  return layout(H, D, r, nullptr, nullptr);
}

int ffn_lopa_approx(int H, int D, int r, const float* w, int max_iters, int32_t* g_idx, int8_t* g_sign,
                    float* lopa_b, float* lopa_a, int* iters, double* objective, void* ws, size_t ws_bytes,
                    hipStream_t stream) {
  if (!w || !g_idx || !g_sign || !lopa_b || !lopa_a || !iters || !objective || !ws) return FFN_ERR_NULL;
  if (!shape_ok(H, D, r)) return FFN_ERR_SHAPE;
  if (max_iters < 1) return FFN_ERR_OPTION;
  if (!aligned16(w) || !aligned16(g_idx) || (reinterpret_cast<uintptr_t>(g_sign) & 3u) || !aligned16(lopa_b) ||
      !aligned16(lopa_a) || !aligned16(ws))
    return FFN_ERR_ALIGN;
  if (ws_bytes < layout(H, D, r, nullptr, nullptr)) return FFN_ERR_WORKSPACE;
  Ws o;
  layout(H, D, r, ws, &o);
  Handle hd;
  if (rocblas_create_handle(&hd.h) != rocblas_status_success) return FFN_ERR_HIP;
  if (rocblas_set_stream(hd.h, stream) != rocblas_status_success) return FFN_ERR_HIP;
  const size_t HD = (size_t)H * D;
  const double one = 1.0, zero = 0.0, minus = -1.0;
  auto hip_ok = [] { return hipGetLastError() == hipSuccess; };

  // U = V = 0: the first M step reads W itself
  k_w_minus_m<<<grid_for(HD), kThreads, 0, stream>>>(w, nullptr, nullptr, o.R, H, D);
  k_m_step<<<H, kThreads, 0, stream>>>(o.R, D, nullptr, nullptr, o.idx[0], o.sgn[0], o.part, o.flags);
  if (!hip_ok()) return FFN_ERR_HIP;
  int cur = 0, done = 0;
  for (int it = 0; it < max_iters; ++it) {
    // UV step: truncated SVD of W - M
    k_w_minus_m<<<grid_for(HD), kThreads, 0, stream>>>(w, o.idx[cur], o.sgn[cur], o.R, H, D);
    if (!hip_ok()) return FFN_ERR_HIP;
    if (rocblas_dsyrk(hd.h, rocblas_fill_lower, rocblas_operation_none, D, H, &one, o.R, D, &zero, o.G, D) !=
        rocblas_status_success)
      return FFN_ERR_HIP;
    if (rocsolver_dsyevd(hd.h, rocblas_evect_original, rocblas_fill_lower, D, o.G, D, o.eig, o.E, o.flags + 1) !=
        rocblas_status_success)
      return FFN_ERR_HIP;
    k_top_vectors<<<grid_for((size_t)r * D), kThreads, 0, stream>>>(o.G, D, r, o.V);
    if (!hip_ok()) return FFN_ERR_HIP;
    // U^T (r x H) = V Ac: V row-major [r][D] is Vc = V^T, D x r column-major
    if (rocblas_dgemm(hd.h, rocblas_operation_transpose, rocblas_operation_none, r, H, D, &one, o.V, D, o.R, D, &zero,
                      o.Ut, r) != rocblas_status_success)
      return FFN_ERR_HIP;
    // residual W - U V: Rc = Wc - Vc Ut
    k_w_minus_m<<<grid_for(HD), kThreads, 0, stream>>>(w, nullptr, nullptr, o.R, H, D);
    if (!hip_ok()) return FFN_ERR_HIP;
    if (rocblas_dgemm(hd.h, rocblas_operation_none, rocblas_operation_none, D, H, r, &minus, o.V, D, o.Ut, r, &one,
                      o.R, D) != rocblas_status_success)
      return FFN_ERR_HIP;
    // M step
    if (hipMemsetAsync(o.flags, 0, sizeof(int), stream) != hipSuccess) return FFN_ERR_HIP;
    k_m_step<<<H, kThreads, 0, stream>>>(o.R, D, o.idx[cur], o.sgn[cur], o.idx[cur ^ 1], o.sgn[cur ^ 1], o.part,
                                         o.flags);
    if (!hip_ok()) return FFN_ERR_HIP;
    int fl[2] = {0, 0};
    if (hipMemcpyAsync(fl, o.flags, sizeof fl, hipMemcpyDeviceToHost, stream) != hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess)
      return FFN_ERR_HIP;
    if (fl[1] != 0) return FFN_ERR_HIP;  // the eigensolver did not converge
    cur ^= 1;
    done = it + 1;
    if (!fl[0]) break;
  }
  k_sum<<<1, kThreads, 0, stream>>>(o.part, H, o.total);
  k_copy_m<<<grid_for((size_t)H), kThreads, 0, stream>>>(o.idx[cur], o.sgn[cur], g_idx, g_sign, H);
  k_to_f32<<<grid_for((size_t)H * r), kThreads, 0, stream>>>(o.Ut, lopa_b, (size_t)H * r);
  k_to_f32<<<grid_for((size_t)r * D), kThreads, 0, stream>>>(o.V, lopa_a, (size_t)r * D);
  if (!hip_ok()) return FFN_ERR_HIP;
  double tot = 0.0;
  if (hipMemcpyAsync(&tot, o.total, sizeof tot, hipMemcpyDeviceToHost, stream) != hipSuccess ||
      hipStreamSynchronize(stream) != hipSuccess)
    return FFN_ERR_HIP;
  *iters = done;
  *objective = tot;
  return FFN_OK;
}

}  // extern "C"
