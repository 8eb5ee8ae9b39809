// Offline spectra of the scored weight matrices (fp64): the Gram matrix of the short
// side and a Householder reduction of that symmetric matrix to tridiagonal form.  The
// eigenvalues of the tridiagonal matrix are the squared singular values the spectral
// concentration ratio needs; they are computed on the host.
#include "common.h"
#include "kernels.h"

namespace sgd {

// ---------------------------------------------------------------------------- Gram
// G[i][j] = sum_t E(t, i) E(t, j) with E(t, i) = X[t][i] (trans = 0) or X[i][t] (trans = 1).
// 64 x 64 output tiles on and below the diagonal; each is mirrored on store.
template <typename T>
__device__ __forceinline__ double ld64(const T* p) { return (double)ElemIO<T>::load(p); }

template <typename T>
__global__ __launch_bounds__(256) void gram_kernel(const T* X, long rows, long cols, int trans, double* G,
                                                   int n, int ntile) {
    constexpr int TB = 64, KB = 16;
    __shared__ double si[KB][TB + 1];
    __shared__ double sj[KB][TB + 1];
    // lower-triangle tile index -> (ti, tj), tj <= ti
    int idx = blockIdx.x, ti = 0;
    while (idx >= ti + 1) { idx -= ti + 1; ++ti; }
    const int tj = idx;
    const int i0 = ti * TB, j0 = tj * TB;
    const long tlen = trans ? cols : rows;
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    double acc[4][4] = {};
    for (long t0 = 0; t0 < tlen; t0 += KB) {
        __syncthreads();
        for (int e = tid; e < KB * TB; e += 256) {
            int kk, c;
            if (trans) { c = e / KB; kk = e % KB; }  // consecutive threads walk t (contiguous in X)
            else { kk = e / TB; c = e % TB; }       // consecutive threads walk i (contiguous in X)
            const long t = t0 + kk;
            const int gi = i0 + c, gj = j0 + c;
            double vi = 0.0, vj = 0.0;
            if (t < tlen) {
                if (gi < n) vi = trans ? ld64(X + (long)gi * cols + t) : ld64(X + t * cols + gi);
                if (gj < n) vj = trans ? ld64(X + (long)gj * cols + t) : ld64(X + t * cols + gj);
            }
            si[kk][c] = vi;
            sj[kk][c] = vj;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < KB; ++kk) {
            double a[4], b[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) a[r] = si[kk][ty + 16 * r];
#pragma unroll
            for (int c = 0; c < 4; ++c) b[c] = sj[kk][tx + 16 * c];
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int c = 0; c < 4; ++c) acc[r][c] = fma(a[r], b[c], acc[r][c]);
        }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int gi = i0 + ty + 16 * r, gj = j0 + tx + 16 * c;
            if (gi < n && gj < n) {
                G[(long)gi * n + gj] = acc[r][c];
                G[(long)gj * n + gi] = acc[r][c];
            }
        }
}

hipError_t launch_gram(int dtype, const void* X, long rows, long cols, int trans, double* G, hipStream_t st) {
    const int n = (int)(trans ? rows : cols);
    const int nt = (n + 63) / 64;
    const int tiles = nt * (nt + 1) / 2;
    if (dtype == 1)
        hipLaunchKernelGGL(gram_kernel<bf16>, dim3(tiles), dim3(256), 0, st, (const bf16*)X, rows, cols, trans, G,
                           n, nt);
    else
        hipLaunchKernelGGL(gram_kernel<float>, dim3(tiles), dim3(256), 0, st, (const float*)X, rows, cols, trans,
                           G, n, nt);
    return hipGetLastError();
}

__global__ void diag_copy_kernel(const double* A, int n, double* out) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
        out[i] = A[(long)i * n + i];
}

hipError_t launch_diag_copy(const double* A, int n, double* out, hipStream_t st) {
    hipLaunchKernelGGL(diag_copy_kernel, dim3((n + 255) / 256), dim3(256), 0, st, A, n, out);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------- tridiagonal
// Householder reduction A = Q T Q^T (Golub & Van Loan, Sec. 8.3.1).  Step j reflects the
// column x = A[j+1:, j] onto beta e_1 with H = I - tau v v^T (v_0 = 1), using the trailing
// block A22 = A[j+1:, j+1:]:  p = tau A22 v,  w = p - (tau/2)(p.v) v,  A22 -= v w^T + w v^T.
// Per step: one single-workgroup kernel (w, the next column, the next reflector) and one
// wide kernel that applies the rank-2 update and, in the same pass, forms the next p.
//
// work layout (doubles): v[2][n] (ping-pong), w[n], p[n], scal[8]: tau[2], ...

constexpr int kHouseThreads = 1024;

__device__ double block_sum_d(double v, double* red) {
    v = warp_sum(v);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    __syncthreads();
    if (lane == 0) red[w] = v;
    __syncthreads();
    double t = 0.0;
    const int nw = blockDim.x >> 6;
    for (int i = 0; i < nw; ++i) t += red[i];
    __syncthreads();
    return t;
}

// Reflector of x[0..len-1] (len >= 1) into vout (vout[0] = 1); returns tau, writes beta.
__device__ double house(const double* x, int len, double* vout, double* beta_out, double* red) {
    double s = 0.0;
    for (int i = 1 + threadIdx.x; i < len; i += blockDim.x) s += x[i] * x[i];
    const double sigma = block_sum_d(s, red);
    const double alpha = x[0];
    double tau, beta, scale;
    if (sigma == 0.0) {
        tau = 0.0;
        beta = alpha;
        scale = 0.0;
    } else {
        const double mu = sqrt(alpha * alpha + sigma);
        beta = alpha <= 0.0 ? mu : -mu;
        tau = (beta - alpha) / beta;
        scale = 1.0 / (alpha - beta);
    }
    for (int i = threadIdx.x; i < len; i += blockDim.x) vout[i] = i == 0 ? 1.0 : x[i] * scale;
    *beta_out = beta;
    return tau;
}

// first reflector (step 0): x = A[0][1..n-1] (row 0 == column 0)
__global__ __launch_bounds__(kHouseThreads) void tri_init_kernel(const double* A, int n, double* v0,
                                                                 double* scal, double* diag, double* offd) {
    __shared__ double red[16];
    double beta;
    const double tau = house(A + 1, n - 1, v0, &beta, red);
    if (threadIdx.x == 0) {
        scal[0] = tau;
        diag[0] = A[0];
        offd[0] = beta;
    }
}

// p = tau A22 v for step 0 (A22 = A[1:, 1:]); one wave per row
__global__ __launch_bounds__(256) void tri_symv0_kernel(const double* A, int n, const double* v,
                                                        const double* scal, double* p) {
    const int m = n - 1;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (row >= m) return;
    const double* ar = A + (long)(1 + row) * n + 1;
    double acc = 0.0;
    for (int c = lane; c < m; c += 64) acc += ar[c] * v[c];
    acc = warp_sum(acc);
    if (lane == 0) p[row] = scal[0] * acc;
}

// Step j: w = p - (tau/2)(p.v) v; the updated column j+1; the next reflector.
__global__ __launch_bounds__(kHouseThreads) void tri_w_house_kernel(const double* A, int n, int j,
                                                                    const double* v, double* vnext,
                                                                    const double* p, double* w, double* xbuf,
                                                                    double* scal, double* diag, double* offd) {
    __shared__ double red[16];
    const int m = n - j - 1;  // size of A22
    const double tau = scal[j & 1];
    double s = 0.0;
    for (int i = threadIdx.x; i < m; i += blockDim.x) s += p[i] * v[i];
    const double pv = block_sum_d(s, red);
    const double k = 0.5 * tau * pv;
    for (int i = threadIdx.x; i < m; i += blockDim.x) w[i] = p[i] - k * v[i];
    __syncthreads();
    const double* arow = A + (long)(j + 1) * n + (j + 1);  // row 0 of A22 (== column 0)
    if (m == 2) {
        // last step: the trailing 2 x 2 block after its update is the end of T
        if (threadIdx.x == 0) {
            diag[j + 1] = arow[0] - 2.0 * v[0] * w[0];
            offd[j + 1] = arow[1] - v[1] * w[0] - w[1] * v[0];
            diag[j + 2] = A[(long)(j + 2) * n + (j + 2)] - 2.0 * v[1] * w[1];
        }
        return;
    }
    // updated column 0 of A22 below the diagonal: x'[i] = A22[1+i][0] - v[1+i] w[0] - w[1+i] v[0]
    for (int i = threadIdx.x; i < m - 1; i += blockDim.x) xbuf[i] = arow[1 + i] - v[1 + i] * w[0] - w[1 + i] * v[0];
    __syncthreads();
    double beta;
    const double taun = house(xbuf, m - 1, vnext, &beta, red);
    if (threadIdx.x == 0) {
        diag[j + 1] = arow[0] - 2.0 * v[0] * w[0];
        offd[j + 1] = beta;
        scal[(j + 1) & 1] = taun;
    }
}

// Step j: A22[i][c] -= v[i] w[c] + w[i] v[c] for i, c >= 1, and the next p:
// pnext[i-1] = tau' sum_{c >= 1} A22[i][c] vnext[c-1].  One wave per row.
__global__ __launch_bounds__(256) void tri_update_kernel(double* A, int n, int j, const double* v,
                                                         const double* w, const double* vnext, const double* scal,
                                                         double* pnext) {
    const int m = n - j - 1;
    const int i = 1 + blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (i >= m) return;
    double* ar = A + (long)(j + 1 + i) * n + (j + 1);
    const double vi = v[i], wi = w[i];
    double acc = 0.0;
    for (int c = 1 + lane; c < m; c += 64) {
        const double a = ar[c] - (vi * w[c] + wi * v[c]);
        ar[c] = a;
        acc += a * vnext[c - 1];
    }
    acc = warp_sum(acc);
    if (lane == 0) pnext[i - 1] = scal[(j + 1) & 1] * acc;
}

hipError_t launch_tridiagonalize(double* A, int n, double* diag, double* offd, double* work, hipStream_t st) {
    if (n == 1) {
        hipMemcpyAsync(diag, A, sizeof(double), hipMemcpyDeviceToDevice, st);
        return hipGetLastError();
    }
    if (n == 2) {
        hipLaunchKernelGGL(diag_copy_kernel, dim3(1), dim3(64), 0, st, A, n, diag);
        hipMemcpyAsync(offd, A + 2, sizeof(double), hipMemcpyDeviceToDevice, st);
        return hipGetLastError();
    }
    double* v[2] = {work, work + n};
    double* w = work + 2 * n;
    double* p = work + 3 * n;
    double* xbuf = work + 4 * n;
    double* scal = work + 5 * n;
    hipLaunchKernelGGL(tri_init_kernel, dim3(1), dim3(kHouseThreads), 0, st, A, n, v[0], scal, diag, offd);
    hipLaunchKernelGGL(tri_symv0_kernel, dim3((n - 1 + 3) / 4), dim3(256), 0, st, A, n, v[0], scal, p);
    for (int j = 0; j <= n - 3; ++j) {
        const int m = n - j - 1;
        hipLaunchKernelGGL(tri_w_house_kernel, dim3(1), dim3(kHouseThreads), 0, st, A, n, j, v[j & 1],
                           v[(j + 1) & 1], p, w, xbuf, scal, diag, offd);
        if (m > 2)
            hipLaunchKernelGGL(tri_update_kernel, dim3((m - 1 + 3) / 4), dim3(256), 0, st, A, n, j, v[j & 1], w,
                               v[(j + 1) & 1], scal, p);
    }
    return hipGetLastError();
}

}  // namespace sgd
