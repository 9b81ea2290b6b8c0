// Depthwise convolution (MobileNetV2's 3x3 filters) on the vector ALU.
//
// Output channel c reads only input channel c, so the node is a per-element
// chain of kh*kw fused multiply-adds: memory-bound, no contraction for the
// matrix cores.  Each element's chain runs over the kh*kw taps in (dy, dx)
// order, starting from 0 (a tap outside the image multiplies a zero input),
// then adds the bias -- the same chain in the full kernel and in the
// channel-list (delta) kernel, so a delta is bit-identical to the full node.
// The full kernel moves 16-byte channel vectors (8 bf16 or 4 fp32 channels of
// one pixel), issuing all taps' loads before the arithmetic; the block's slot
// weights sit in LDS as fp32, tap-major, so a lane's channels are contiguous.
#include "dev.hpp"

namespace mure {

namespace {
constexpr int DW_MAXW = 8192;                         // C * kh * kw staged in LDS
constexpr int DW_MAXC = 2048;
}

// zeros that taps outside the image read instead of the input
static __device__ __attribute__((aligned(16))) v4u g_dw_zero[1] = {};

// KH, KW: the filter size when known at compile time (3 x 3), else 0.  The
// block's LDS (dynamic, sized to the node) holds the slot's weights [tap][C]
// and bias; each thread takes work items it and it + 256 of every 512 and
// requests both items' tap vectors before their arithmetic.
template <typename T, int KH, int KW>
__global__ __launch_bounds__(256) void dw_full_kernel(DwArgs a, int rows, DivU32 dcv, DivU32 dpix,
                                                      DivU32 dwo) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int NT = KH * KW > 0 ? KH * KW : 1, KWC = KW > 0 ? KW : 1;
  extern __shared__ __attribute__((aligned(16))) float dw_lds[];
  const int tid = threadIdx.x;
  const int sl = a.slot0 + (int)blockIdx.y;
  const int kh = KH ? KH : a.kh, kw = KW ? KW : a.kw;
  const int taps = kh * kw;
  float* const wl = dw_lds;                           // [tap][C]
  float* const bl = dw_lds + a.C * taps;              // [C]
  const T* __restrict__ Wt = reinterpret_cast<const T*>(a.wtab[sl]);
  for (int e = tid; e < a.C * taps; e += 256) {
    const int c = e / taps, tp = e - c * taps;
    wl[tp * a.C + c] = to_f<T>(Wt[e]);
  }
  for (int c = tid; c < a.C; c += 256) bl[c] = a.btab[sl][c];
  __syncthreads();
  const v4u* const zp = reinterpret_cast<const v4u*>(g_dw_zero);
  const int xi0 = (int)blockIdx.x * rows;
  const int nr = min(rows, a.nx - xi0);
  const int per = a.Ho * a.Wo * (a.C / VEC);          // vectors per output row
  const int total = nr * per;
  const T* __restrict__ X = reinterpret_cast<const T*>(a.in.p);

  // one work item: output vector (input ii, pixel, channel vector cv)
  struct Item {
    int cv, pix;
    int64_t r;
    v4u xv[NT];
  };
  auto request = [&](Item& w, int it) {
    int ii, rem, oy, ox;
    divmodu(dpix, (uint32_t)it, ii, rem);             // rem = pixel * (C / VEC) + cv
    divmodu(dcv, (uint32_t)rem, w.pix, w.cv);
    divmodu(dwo, (uint32_t)w.pix, oy, ox);
    w.r = (int64_t)sl * a.nx + xi0 + ii;
    const T* xr = X + row_index(a.in.mode, w.r, a.nx, a.x0) * a.in.row_elems + w.cv * VEC;
    const int iy0 = oy * a.stride - a.pad, ix0 = ox * a.stride - a.pad;
#pragma unroll
    for (int tp = 0; tp < NT; ++tp) {
      const int iy = iy0 + tp / KWC, ix = ix0 + tp % KWC;
      const bool ok = (unsigned)iy < (unsigned)a.H && (unsigned)ix < (unsigned)a.W;
      w.xv[tp] = *(ok ? reinterpret_cast<const v4u*>(xr + ((int64_t)iy * a.W + ix) * a.C) : zp);
    }
  };
  auto finish = [&](const Item& w) {
    // the chains in (dy, dx) order from 0, then the bias
    float acc[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) acc[j] = 0.f;
#pragma unroll
    for (int tp = 0; tp < NT; ++tp) {
      T x8[VEC];
      __builtin_memcpy(x8, &w.xv[tp], 16);
      const float* wt = wl + tp * a.C + w.cv * VEC;
#pragma unroll
      for (int j = 0; j < VEC; ++j) acc[j] = fmaf(to_f<T>(x8[j]), wt[j], acc[j]);
    }
    T ov[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) ov[j] = from_f<T>(act(acc[j] + bl[w.cv * VEC + j], a.relu));
    v4u o;
    __builtin_memcpy(&o, ov, 16);
    const int64_t ro = row_index(a.out_mode, w.r, a.nx, a.x0);
    *reinterpret_cast<v4u*>(reinterpret_cast<T*>(a.out) + ro * a.out_row + (int64_t)w.pix * a.C + w.cv * VEC) = o;
  };

  if constexpr (KH > 0) {
    for (int base = 0; base < total; base += 512) {
      const int i0 = base + tid, i1 = base + 256 + tid;
      Item w0, w1;
      if (i0 < total) request(w0, i0);
      if (i1 < total) request(w1, i1);
      if (i0 < total) finish(w0);
      if (i1 < total) finish(w1);
    }
  } else {
    for (int it = tid; it < total; it += 256) {
      int ii, rem, pix, cv, oy, ox;
      divmodu(dpix, (uint32_t)it, ii, rem);
      divmodu(dcv, (uint32_t)rem, pix, cv);
      divmodu(dwo, (uint32_t)pix, oy, ox);
      const int64_t r = (int64_t)sl * a.nx + xi0 + ii;
      const T* xr = X + row_index(a.in.mode, r, a.nx, a.x0) * a.in.row_elems + cv * VEC;
      const int iy0 = oy * a.stride - a.pad, ix0 = ox * a.stride - a.pad;
      float acc[VEC];
#pragma unroll
      for (int j = 0; j < VEC; ++j) acc[j] = 0.f;
      for (int tp = 0; tp < taps; ++tp) {
        const int iy = iy0 + tp / kw, ix = ix0 + tp % kw;
        const bool ok = (unsigned)iy < (unsigned)a.H && (unsigned)ix < (unsigned)a.W;
        const v4u raw = *(ok ? reinterpret_cast<const v4u*>(xr + ((int64_t)iy * a.W + ix) * a.C) : zp);
        T x8[VEC];
        __builtin_memcpy(x8, &raw, 16);
        const float* wt = wl + tp * a.C + cv * VEC;
#pragma unroll
        for (int j = 0; j < VEC; ++j) acc[j] = fmaf(to_f<T>(x8[j]), wt[j], acc[j]);
      }
      T ov[VEC];
#pragma unroll
      for (int j = 0; j < VEC; ++j) ov[j] = from_f<T>(act(acc[j] + bl[cv * VEC + j], a.relu));
      v4u o;
      __builtin_memcpy(&o, ov, 16);
      const int64_t ro = row_index(a.out_mode, r, a.nx, a.x0);
      *reinterpret_cast<v4u*>(reinterpret_cast<T*>(a.out) + ro * a.out_row + (int64_t)pix * a.C + cv * VEC) = o;
    }
  }
}

// 3 x 3 filters: each thread walks one (input, output column, channel vector)
// down the image with the three input rows of the current output row in
// registers, so a new output row loads only the rows it does not share with
// the previous one (one for stride 1, two for stride 2), requested before the
// current row's arithmetic.  The chains are the full kernel's: taps in (dy, dx)
// order from 0, then the bias.  No LDS: a thread's filters come from global
// memory once.  In bf16 they stay packed in registers and are widened at
// each use (127 and 151 VGPRs for stride 1 and 2, four and three waves per
// SIMD, against 176 and 200 with the widened filters held: two).
template <typename T, int S>
__global__ __launch_bounds__(256, sizeof(T) == 2 ? 3 : 1) void dw_col_kernel(DwArgs a, int tasks, DivU32 dcv, DivU32 dwo) {
  constexpr int VEC = 16 / sizeof(T);
  constexpr int NNEW = S == 1 ? 1 : 2;                 // new input rows per output row
  const int sl = a.slot0 + (int)blockIdx.y;
  const int t = (int)blockIdx.x * 256 + (int)threadIdx.x;
  if (t >= tasks) return;
  int rest, cv, xi, ox;
  divmodu(dcv, (uint32_t)t, rest, cv);                 // t = (xi * Wo + ox) * (C / VEC) + cv
  divmodu(dwo, (uint32_t)rest, xi, ox);
  const int64_t r = (int64_t)sl * a.nx + xi;
  const T* __restrict__ xr = reinterpret_cast<const T*>(a.in.p) +
                             row_index(a.in.mode, r, a.nx, a.x0) * a.in.row_elems + cv * VEC;
  T* const orow = reinterpret_cast<T*>(a.out) + row_index(a.out_mode, r, a.nx, a.x0) * a.out_row + cv * VEC;
  // the thread's channels' filters ([C][3][3]: VEC * 9 consecutive elements),
  // kept in the node type and widened at each use, and biases, straight from
  // global memory (L2-resident, shared by every column of the slot)
  v4u wraw[9];
  float b[VEC];
  {
    const T* __restrict__ wsrc = reinterpret_cast<const T*>(a.wtab[sl]) + (int64_t)cv * VEC * 9;
#pragma unroll
    for (int q = 0; q < 9; ++q) wraw[q] = reinterpret_cast<const v4u*>(wsrc)[q];
    const float* __restrict__ bsrc = a.btab[sl] + cv * VEC;
#pragma unroll
    for (int j = 0; j < VEC; ++j) b[j] = bsrc[j];
  }
  const int ix0 = ox * S - a.pad;
  bool colok[3];
#pragma unroll
  for (int dx = 0; dx < 3; ++dx) colok[dx] = (unsigned)(ix0 + dx) < (unsigned)a.W;
  // the three vectors of input row iy under this column (zeros outside the image)
  auto load_row = [&](int iy, v4u* v) {
#pragma unroll
    for (int dx = 0; dx < 3; ++dx)
      v[dx] = (unsigned)iy < (unsigned)a.H && colok[dx]
                  ? *reinterpret_cast<const v4u*>(xr + ((int64_t)iy * a.W + ix0 + dx) * a.C)
                  : v4u{0u, 0u, 0u, 0u};
  };
  // window rows[3] of the current output row; the new rows of the next two
  // output rows (nr1, nr2: one row each for stride 1, two for stride 2) are in
  // flight meanwhile
  v4u row[3][3], nr1[NNEW][3], nr2[NNEW][3];
  load_row(-a.pad, row[0]);
  load_row(-a.pad + 1, row[1]);
  load_row(-a.pad + 2, row[2]);
#pragma unroll
  for (int k = 0; k < NNEW; ++k) load_row(S - a.pad + 3 - NNEW + k, nr1[k]);
  for (int oy = 0; oy < a.Ho; ++oy) {
    const int iy2 = (oy + 2) * S - a.pad + 3 - NNEW;  // first new row of output row oy + 2
#pragma unroll
    for (int k = 0; k < NNEW; ++k) load_row(iy2 + k, nr2[k]);
    // the filters stay packed across rows: hoisting their widening out of
    // the row loop would hold them as VEC * 9 floats
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int q = 0; q < 9; ++q) asm volatile("" : "+v"(wraw[q]));
    }
    T wv[VEC * 9];
    __builtin_memcpy(wv, wraw, sizeof(wv));
    float acc[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) acc[j] = 0.f;
#pragma unroll
    for (int dy = 0; dy < 3; ++dy)
#pragma unroll
      for (int dx = 0; dx < 3; ++dx) {
        T x8[VEC];
        __builtin_memcpy(x8, &row[dy][dx], 16);
#pragma unroll
        for (int j = 0; j < VEC; ++j) acc[j] = fmaf(to_f<T>(x8[j]), to_f<T>(wv[j * 9 + dy * 3 + dx]), acc[j]);
      }
    T ov[VEC];
#pragma unroll
    for (int j = 0; j < VEC; ++j) ov[j] = from_f<T>(act(acc[j] + b[j], a.relu));
    v4u o;
    __builtin_memcpy(&o, ov, 16);
    *reinterpret_cast<v4u*>(orow + ((int64_t)oy * a.Wo + ox) * a.C) = o;
#pragma unroll
    for (int dx = 0; dx < 3; ++dx) {
      if constexpr (S == 1) {
        row[0][dx] = row[1][dx];
        row[1][dx] = row[2][dx];
        row[2][dx] = nr1[0][dx];
      } else {
        row[0][dx] = row[2][dx];
        row[1][dx] = nr1[0][dx];
        row[2][dx] = nr1[1][dx];
      }
#pragma unroll
      for (int k = 0; k < NNEW; ++k) nr1[k][dx] = nr2[k][dx];
    }
  }
}

// One element per thread: (input, pixel, listed channel).  Used for the delta
// channel lists, for C % 16-byte-vector != 0, and for float32 network outputs.
template <typename T>
__global__ __launch_bounds__(256) void dw_list_kernel(DwArgs a, int rows, DivU32 dwo) {
  const int tid = threadIdx.x;
  const int sl = a.slot0 + (int)blockIdx.y;
  int c_beg = 0, c_end = a.C;
  if (a.ch_off) { c_beg = a.ch_off[sl]; c_end = a.ch_off[sl + 1]; }
  const int nch = c_end - c_beg;
  if (nch <= 0) return;
  const int taps = a.kh * a.kw;
  const T* __restrict__ Wt = reinterpret_cast<const T*>(a.wtab[sl]);
  const float* __restrict__ bias = a.btab[sl];
  const int xi0 = (int)blockIdx.x * rows;
  const int nr = min(rows, a.nx - xi0);
  const int per = a.Ho * a.Wo * nch;
  const T* __restrict__ X = reinterpret_cast<const T*>(a.in.p);
  for (int it = tid; it < nr * per; it += 256) {
    int oy, ox;
    const int ii = it / per, rem = it - ii * per;      // rem = pixel * nch + u
    const int pix = rem / nch, u = rem - pix * nch;
    divmodu(dwo, (uint32_t)pix, oy, ox);
    const int c = a.ch_list ? a.ch_list[c_beg + u] : c_beg + u;
    const int xi = xi0 + ii;
    const int64_t r = (int64_t)sl * a.nx + xi;
    const T* xr = X + row_index(a.in.mode, r, a.nx, a.x0) * a.in.row_elems + c;
    const T* wr = Wt + (int64_t)c * taps;
    float acc = 0.f;
    const int iy0 = oy * a.stride - a.pad, ix0 = ox * a.stride - a.pad;
    for (int dy = 0; dy < a.kh; ++dy) {
      const int iy = iy0 + dy;
      for (int dx = 0; dx < a.kw; ++dx) {
        const int ix = ix0 + dx;
        // taps outside the image contribute a zero input, as in the full kernel
        const bool ok = (unsigned)iy < (unsigned)a.H && (unsigned)ix < (unsigned)a.W;
        const float x = ok ? to_f<T>(xr[((int64_t)iy * a.W + ix) * a.C]) : 0.f;
        acc = fmaf(x, to_f<T>(wr[dy * a.kw + dx]), acc);
      }
    }
    const float v = act(acc + bias[c], a.relu);
    const int64_t ro = row_index(a.out_mode, r, a.nx, a.x0);
    if (a.delta_T > 0) store_out<T>(a.out, 0, ro * a.out_row + (int64_t)pix * a.delta_T + u, v);
    else store_out<T>(a.out, a.out_f32, ro * a.out_row + (int64_t)pix * a.C + c, v);
  }
}

hipError_t launch_dw(const DwArgs& a, int dtype, hipStream_t s) {
  if (a.nslots <= 0 || a.nx <= 0) return hipSuccess;
  if (a.nslots > 65535) return hipErrorInvalidValue;
  const int esize = dtype == 0 ? 4 : 2;
  const int vec = 16 / esize;
  const bool full = !a.ch_off && !a.out_f32 && a.C % vec == 0 && a.C * a.kh * a.kw <= DW_MAXW &&
                    a.C <= DW_MAXC && a.in.row_elems % vec == 0;
  const int64_t pix = (int64_t)a.Ho * a.Wo;
  // about 4K items per block
  const int64_t items_per_row = full ? pix * (a.C / vec) : pix * a.C;
  const int rows = (int)std::max<int64_t>(1, std::min<int64_t>(a.nx, 4096 / std::max<int64_t>(1, items_per_row)));
  if (items_per_row * rows >= INT32_MAX) return hipErrorInvalidValue;
  dim3 grid((unsigned)((a.nx + rows - 1) / rows), (unsigned)a.nslots);
  const DivU32 dwo = make_divu32((uint32_t)a.Wo);
  if (full) {
    const DivU32 dcv = make_divu32((uint32_t)(a.C / vec));
    const DivU32 dpix = make_divu32((uint32_t)(pix * (a.C / vec)));
    const size_t lds = (size_t)a.C * (a.kh * a.kw + 1) * sizeof(float);
    if (a.kh == 3 && a.kw == 3 && (a.stride == 1 || a.stride == 2)) {
      // one task per (input, output column, channel vector)
      const int64_t tasks = (int64_t)a.nx * a.Wo * (a.C / vec);
      if (tasks >= INT32_MAX) return hipErrorInvalidValue;
      dim3 g2((unsigned)((tasks + 255) / 256), (unsigned)a.nslots);
      if (dtype == 0 && a.stride == 1) hipLaunchKernelGGL((dw_col_kernel<float, 1>), g2, dim3(256), 0, s, a, (int)tasks, dcv, dwo);
      else if (dtype == 0) hipLaunchKernelGGL((dw_col_kernel<float, 2>), g2, dim3(256), 0, s, a, (int)tasks, dcv, dwo);
      else if (a.stride == 1) hipLaunchKernelGGL((dw_col_kernel<bf16_t, 1>), g2, dim3(256), 0, s, a, (int)tasks, dcv, dwo);
      else hipLaunchKernelGGL((dw_col_kernel<bf16_t, 2>), g2, dim3(256), 0, s, a, (int)tasks, dcv, dwo);
    } else if (dtype == 0) {
      hipLaunchKernelGGL((dw_full_kernel<float, 0, 0>), grid, dim3(256), lds, s, a, rows, dcv, dpix, dwo);
    } else {
      hipLaunchKernelGGL((dw_full_kernel<bf16_t, 0, 0>), grid, dim3(256), lds, s, a, rows, dcv, dpix, dwo);
    }
  } else {
    // the row split assumes every channel (the largest list)
    if (dtype == 0) hipLaunchKernelGGL(dw_list_kernel<float>, grid, dim3(256), 0, s, a, rows, dwo);
    else hipLaunchKernelGGL(dw_list_kernel<bf16_t>, grid, dim3(256), 0, s, a, rows, dwo);
  }
  return hipGetLastError();
}

}  // namespace mure
