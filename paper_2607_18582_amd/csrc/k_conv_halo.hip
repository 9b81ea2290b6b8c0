// bf16 3x3 convolutions with stride 1 and padding 1 (C_in % 16 == 0, image
// width 8, 16, 32 or 64) as an implicit GEMM on MFMA whose operands both come
// from LDS (v_mfma_f32_16x16x32_bf16).
//
// Block tile: 512 output pixels x BN output channels, eight waves of 64 rows
// (one block per CU: the LDS stages below take most of it).  The pixels are
// TR = 512 / W consecutive image rows -- a band of one image, or 512 / (H W)
// whole images -- so a tile never mixes two images' borders.
// The input channels go in chunks of 16.  Per chunk the block stages in LDS
// (a) the band's input rows plus a one-pixel border (the halo, zero outside
// the image): every input element crosses the memory pipeline once per block
// and chunk instead of once per tap as an im2col gather would; and (b) the
// chunk's weights for the tile's columns.  One MFMA k-step of 32 covers two
// taps of the chunk (taps 2p and 2p+1; a tenth, all-zero tap pads the
// ninth), so a chunk is five k-steps.  The stages are double-buffered in LDS
// and fetched into registers two chunks ahead: the k loop has one barrier per
// chunk and no global loads of its own.
//
// Reduction order: k = (chunk of 16 channels, tap pair, tap, channel), fixed
// for a node shape; every launch of a node (full rows or gathered delta
// columns) uses it.
#include "dev.hpp"
#include "plan.hpp"

namespace mure {

namespace {
constexpr int HALO_PS = 24;                            // LDS pixel stride: 16 channels + 8 (bf16)
constexpr int HALO_ELEMS = HALO_MAXPX * HALO_PS;       // halo part of a stage (elements)
typedef __attribute__((address_space(1))) const v4u gv4u;
}

// Zero bytes that out-of-image halo pixels and the padding tap read.
static __device__ __attribute__((aligned(16))) v4u g_halo_zero[4] = {};

template <int W, int BN>
__global__ __launch_bounds__(512)
void conv_halo_kernel(ConvArgs a) {
  constexpr int NT = 512, BM = 512, TR = BM / W, W2 = W + 2;
  constexpr int TM = 4, TN = BN / 16;                  // a wave: 64 rows x BN columns
  constexpr int B_ELEMS = 5 * BN * 32;                 // weight part of a stage: [pair][column][32]
  constexpr int STAGE = HALO_ELEMS + B_ELEMS;
  constexpr int OLD = BN + 8;                          // staged output row (bf16)
  constexpr int LDS_ELEMS = 2 * STAGE > BM * OLD ? 2 * STAGE : BM * OLD;
  constexpr int HV = (HALO_MAXPX * 2 + NT - 1) / NT;   // halo vectors per thread and chunk
  constexpr int BV = (5 * BN * 4 + NT - 1) / NT;       // weight vectors per thread and chunk
  __shared__ __attribute__((aligned(16))) bf16_t smem[LDS_ELEMS];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int slot = a.slot0 + (int)blockIdx.y;
  // XCD-aware order: consecutive blocks go round-robin to the 8 XCDs, so block
  // b runs on XCD b % 8; the column blocks of one band take consecutive turns
  // on the same XCD and share its L2 copy of the band's input
  const int bx = (int)blockIdx.x, xcd = bx & 7, turn = bx >> 3;
  const int band = (turn / a.zblocks) * 8 + xcd;
  if (band >= a.bands) return;                           // padding of the order (whole block)
  const int n0 = (turn % a.zblocks) * BN;
  const int ncol = a.cols ? a.ncols : a.Cout;
  // the band: image rows [r0, r0 + TR) of the flattened (input, row) axis;
  // RI rows of each of IMGS images (RI = H when whole images are packed)
  const int RI = a.H < TR ? a.H : TR;
  const int IMGS = TR / RI;
  const int64_t r0 = (int64_t)band * TR;
  const int xi0 = (int)(r0 / a.H), y0 = (int)(r0 % a.H);
  const int npx = IMGS * (RI + 2) * W2;                // halo pixels (<= HALO_MAXPX, checked by the launcher)
  const bf16_t* const zp = reinterpret_cast<const bf16_t*>(g_halo_zero);

  // halo vectors of this thread: vector v = tid + NT j is pixel v / 2,
  // channels (v % 2) * 8 .. + 8 of the chunk, at element offset hoff[j] from
  // the band's first input row (consecutive inputs are consecutive rows in
  // both tensor modes); -1 reads zeros, -2 is past the halo (not stored)
  const bf16_t* const in0 = reinterpret_cast<const bf16_t*>(a.in.p) +
                            row_index(a.in.mode, (int64_t)slot * a.nx + (xi0 < a.nx ? xi0 : 0), a.nx, a.x0) *
                                a.in.row_elems;
  int hoff[HV];
#pragma unroll
  for (int j = 0; j < HV; ++j) {
    const int v = tid + NT * j;
    const int px = v >> 1, h = v & 1;
    hoff[j] = -2;
    if (px < npx) {
      hoff[j] = -1;
      const int im = px / ((RI + 2) * W2), rem = px % ((RI + 2) * W2);
      const int hy = rem / W2, hx = rem % W2;
      const int y = y0 + hy - 1, x = hx - 1;
      if (xi0 + im < a.nx && (unsigned)y < (unsigned)a.H && (unsigned)x < (unsigned)W)
        hoff[j] = (int)(im * a.in.row_elems) + (y * W + x) * a.C + h * 8;
    }
  }
  // weight vectors of this thread: vector v = tid + NT j is tap pair p,
  // column n, quarter q (8 of the pair's 32 k: tap 2p + q / 2, channels
  // (q % 2) * 8 ..); bsrc is its source at chunk 0 (nullptr: zeros), bdst its
  // LDS slot, the quarter rotated by (n / 4) % 4 so that the 16 lanes reading
  // one quarter of 16 consecutive columns hit distinct banks
  const bf16_t* bsrc[BV];
  int bdst[BV];
#pragma unroll
  for (int j = 0; j < BV; ++j) {
    const int v = tid + NT * j;
    const int p = v / (BN * 4), rem = v % (BN * 4);
    const int n = rem >> 2, q = rem & 3;
    const int tap = 2 * p + (q >> 1);
    bsrc[j] = nullptr;
    bdst[j] = -1;
    if (p < 5) {
      bdst[j] = ((p * BN + n) * 4 + (q ^ ((n >> 2) & 3))) * 8;
      const int nc = n0 + n;
      if (tap < 9 && nc < ncol) {
        const bf16_t* row;
        if (a.cols) {
          const DeltaCol cd = a.cols[nc];
          row = reinterpret_cast<const bf16_t*>(a.wtab[a.slot0 + cd.slot - a.col_slot0]) + (int64_t)cd.c * a.K;
        } else {
          row = reinterpret_cast<const bf16_t*>(a.wtab[slot]) + (int64_t)nc * a.K;
        }
        bsrc[j] = row + tap * a.C + (q & 1) * 8;
      }
    }
  }
  // one chunk's staging registers
  struct Regs { v4u h[HV], b[BV]; };
  auto fetch = [&](Regs& r, int c0) {
#pragma unroll
    for (int j = 0; j < HV; ++j) r.h[j] = *(const gv4u*)(hoff[j] >= 0 ? in0 + hoff[j] + c0 : zp);
#pragma unroll
    for (int j = 0; j < BV; ++j) r.b[j] = *(const gv4u*)(bsrc[j] ? bsrc[j] + c0 : zp);
  };
  auto stage = [&](const Regs& r, int buf) {
    bf16_t* st = smem + buf * STAGE;
#pragma unroll
    for (int j = 0; j < HV; ++j) {
      const int v = tid + NT * j;
      if (hoff[j] != -2) *reinterpret_cast<v4u*>(&st[(v >> 1) * HALO_PS + (v & 1) * 8]) = r.h[j];
    }
#pragma unroll
    for (int j = 0; j < BV; ++j)
      if (bdst[j] >= 0) *reinterpret_cast<v4u*>(&st[HALO_ELEMS + bdst[j]]) = r.b[j];
  };

  // A fragment bases: lane row (lane & 15) of M tile i is band pixel m; the
  // lane's 8 k are channels (q % 2) * 8 of tap 2p + q / 2 (q = lane >> 4), so
  // its halo pixel is the pair's first tap shifted by 0 or by the distance to
  // the second tap: 1 pixel (pairs 0, 2, 3), W + 2 - 2 pixels (pair 1: taps
  // 2 and 3 change row), 0 (pair 4: the zero tap, any finite value)
  const int q = lane >> 4;
  int abase0[TM], abase1[TM], abase2[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int m = wave * 64 + i * 16 + (lane & 15);
    const int row = m / W, x = m % W;
    const int im = row / RI, y = row % RI;
    abase0[i] = ((im * (RI + 2) + y) * W2 + x) * HALO_PS + (q & 1) * 8;
    abase1[i] = abase0[i] + (q >> 1) * HALO_PS;
    abase2[i] = abase0[i] + (q >> 1) * (W2 - 2) * HALO_PS;
  }
  // B fragment: column j * 16 + (lane & 15), quarter q, rotated as stored
  const int bbase = ((lane & 15) * 4 + (q ^ ((lane >> 2) & 3))) * 8;

  v4f acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int buf) {
    const bf16_t* st = smem + buf * STAGE;
#pragma unroll
    for (int p = 0; p < 5; ++p) {
      const int t0 = 2 * p;
      const int toff = ((t0 / 3) * W2 + (t0 % 3)) * HALO_PS;
      v8bf av[TM], bv[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int base = p == 1 ? abase2[i] : p == 4 ? abase0[i] : abase1[i];
        av[i] = *reinterpret_cast<const v8bf*>(&st[base + toff]);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bv[j] = *reinterpret_cast<const v8bf*>(&st[HALO_ELEMS + (p * BN + j * 16) * 32 + bbase]);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
  };

  // chunks c = 0 .. nch-1 through buffers c % 2; registers RA / RB hold the
  // chunks two ahead (fetches past the last chunk reload it, unused, so that
  // every path keeps the same requests in flight)
  const int nch = a.C / 16;
  auto cidx = [&](int c) { return (c < nch ? c : nch - 1) * 16; };
  Regs RA, RB;
  fetch(RA, 0);
  stage(RA, 0);
  fetch(RA, cidx(1));
  fetch(RB, cidx(2));
  __syncthreads();
  // pairs of chunks, straight-line (the same requests in flight on every
  // path); past the last chunk the stores write a reloaded chunk nobody reads
  int c = 0;
  for (; c + 1 < nch; c += 2) {
    compute(0);
    stage(RA, 1);
    fetch(RA, cidx(c + 3));
    __syncthreads();
    compute(1);
    stage(RB, 0);
    fetch(RB, cidx(c + 4));
    __syncthreads();
  }
  if (c < nch) compute(0);                             // odd chunk count: the last one
  __syncthreads();

  // ---- epilogue: bias, activation, bf16 rounding, staged in LDS ----
  bf16_t* Os = smem;                                   // [BM][OLD]
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int nl = j * 16 + (lane & 15);
    const int nc = n0 + nl;
    float bv = 0.f;
    if (nc < ncol) {
      if (a.cols) {
        const DeltaCol cd = a.cols[nc];
        bv = a.btab[a.slot0 + cd.slot - a.col_slot0][cd.c];
      } else {
        bv = a.btab[slot][nc];
      }
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        Os[(wave * 64 + i * 16 + (lane >> 4) * 4 + e) * OLD + nl] = f2bf(act(acc[i][j][e] + bv, a.relu));
  }
  __syncthreads();

  // band pixel m -> (input xi, image row y, column x)
  auto pixel = [&](int m, int& xi, int& y, int& x) {
    const int row = m / W;
    x = m % W;
    xi = xi0 + row / RI;
    y = y0 + row % RI;
  };
  if (a.cols) {
    // gathered columns: each column has its own slot and channel
    const int PX = a.pool ? BM / 4 : BM;
    for (int idx = tid; idx < PX * BN; idx += NT) {
      const int nl = idx / PX, p = idx % PX;
      const int nc = n0 + nl;
      if (nc >= ncol) continue;
      int xi, y, x;
      float v;
      if (a.pool) {
        // pooled pixel p: band rows 2 (p / (W/2)) .. +1, columns 2 (p % (W/2)) .. +1
        const int pr = p / (W / 2), pc = p % (W / 2);
        const int m = 2 * pr * W + 2 * pc;
        pixel(m, xi, y, x);
        v = fmaxf(fmaxf(bf2f(Os[m * OLD + nl]), bf2f(Os[(m + 1) * OLD + nl])),
                  fmaxf(bf2f(Os[(m + W) * OLD + nl]), bf2f(Os[(m + W + 1) * OLD + nl])));
        y >>= 1; x >>= 1;
      } else {
        pixel(p, xi, y, x);
        v = bf2f(Os[p * OLD + nl]);
      }
      if (xi >= a.nx) continue;
      const DeltaCol cd = a.cols[nc];
      const int os = a.slot0 + cd.slot - a.col_slot0;
      const int ostride = a.delta_T > 0 ? a.delta_T : a.Cout;
      const int n = a.delta_T > 0 ? cd.t : cd.c;
      const int Wo = a.pool ? W / 2 : W;
      const int64_t ro = row_index(a.out_mode, (int64_t)os * a.nx + xi, a.nx, a.x0);
      reinterpret_cast<bf16_t*>(a.out)[ro * a.out_row + ((int64_t)y * Wo + x) * ostride + n] = f2bf(v);
    }
    return;
  }
  constexpr int VPR = BN / 8;                          // 16-byte vectors per staged row
  if (a.pool) {
    for (int idx = tid; idx < (BM / 4) * VPR; idx += NT) {
      const int p = idx / VPR, vc = idx % VPR;
      const int n = n0 + vc * 8;
      if (n >= a.Cout) continue;
      const int pr = p / (W / 2), pc = p % (W / 2);
      const int m = 2 * pr * W + 2 * pc;
      int xi, y, x;
      pixel(m, xi, y, x);
      if (xi >= a.nx) continue;
      // the max of the rounded values is the rounded max (rounding is monotonic)
      const v4u q0 = *reinterpret_cast<const v4u*>(&Os[m * OLD + vc * 8]);
      const v4u q1 = *reinterpret_cast<const v4u*>(&Os[(m + 1) * OLD + vc * 8]);
      const v4u q2 = *reinterpret_cast<const v4u*>(&Os[(m + W) * OLD + vc * 8]);
      const v4u q3 = *reinterpret_cast<const v4u*>(&Os[(m + W + 1) * OLD + vc * 8]);
      v4u o;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        uint32_t r = 0;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int sh = 16 * h;
          const float f = fmaxf(fmaxf(bf2f((bf16_t)(q0[w] >> sh)), bf2f((bf16_t)(q1[w] >> sh))),
                                fmaxf(bf2f((bf16_t)(q2[w] >> sh)), bf2f((bf16_t)(q3[w] >> sh))));
          r |= (uint32_t)f2bf(f) << sh;
        }
        o[w] = r;
      }
      const int64_t ro = row_index(a.out_mode, (int64_t)slot * a.nx + xi, a.nx, a.x0);
      *reinterpret_cast<v4u*>(reinterpret_cast<bf16_t*>(a.out) + ro * a.out_row +
                              ((int64_t)(y >> 1) * (W / 2) + (x >> 1)) * a.Cout + n) = o;
    }
    return;
  }
  for (int idx = tid; idx < BM * VPR; idx += NT) {
    const int m = idx / VPR, vc = idx % VPR;
    const int n = n0 + vc * 8;
    if (n >= a.Cout) continue;
    int xi, y, x;
    pixel(m, xi, y, x);
    if (xi >= a.nx) continue;
    const int64_t q = (int64_t)y * W + x;
    v4u val = *reinterpret_cast<const v4u*>(&Os[m * OLD + vc * 8]);
    if (a.add_mode) {
      // the rounded convolution + the shortcut, in float32, then the ADD's activation
      const bf16_t* sp = reinterpret_cast<const bf16_t*>(a.skip.p) +
                         row_index(a.skip.mode, (int64_t)slot * a.nx + xi, a.nx, a.x0) * a.skip.row_elems;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        uint32_t o = 0;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int c = n + 2 * w + h;
          float s = 0.f;
          if (a.add_mode == 1) {
            s = bf2f(sp[q * a.Cout + c]);
          } else {
            // option A: the skip subsampled by 2 and zero-padded in channels
            const int cs = c - (a.Cout - a.Cs) / 2;
            if (cs >= 0 && cs < a.Cs) s = bf2f(sp[((int64_t)(2 * y) * a.Ws + 2 * x) * a.Cs + cs]);
          }
          const float t = act(bf2f((bf16_t)(val[w] >> (16 * h))) + s, a.add_relu);
          o |= (uint32_t)f2bf(t) << (16 * h);
        }
        val[w] = o;
      }
    }
    const int64_t ro = row_index(a.out_mode, (int64_t)slot * a.nx + xi, a.nx, a.x0);
    *reinterpret_cast<v4u*>(reinterpret_cast<bf16_t*>(a.out) + ro * a.out_row + q * a.Cout + n) = val;
  }
}

int conv_halo_bn(int cout) { return cout <= 16 ? 16 : cout <= 32 ? 32 : 64; }

template <int W>
static hipError_t launch_halo_w(const ConvArgs& a, dim3 grid, int bn, hipStream_t s) {
  switch (bn) {
    case 16: hipLaunchKernelGGL((conv_halo_kernel<W, 16>), grid, dim3(512), 0, s, a); break;
    case 32: hipLaunchKernelGGL((conv_halo_kernel<W, 32>), grid, dim3(512), 0, s, a); break;
    default: hipLaunchKernelGGL((conv_halo_kernel<W, 64>), grid, dim3(512), 0, s, a); break;
  }
  return hipGetLastError();
}

hipError_t launch_conv_halo(const ConvArgs& a0, int nslots, hipStream_t s) {
  if (nslots <= 0 || a0.nx <= 0) return hipSuccess;
  if (!conv_halo_fits(a0.H, a0.W, a0.C, a0.kh, a0.kw, a0.stride, a0.pad) || a0.Cout % 8 ||
      a0.out_f32 || a0.add_out_f32 || (a0.pool && a0.add_mode) || a0.vin.chmap)
    return hipErrorInvalidValue;
  if (a0.cols && (a0.in.mode != MODE_CACHE || a0.add_mode || a0.ncols <= 0)) return hipErrorInvalidValue;
  ConvArgs a = a0;
  if (a.cols) nslots = 1;
  const int TR = 512 / a.W;
  const int ncol = a.cols ? a.ncols : a.Cout;
  const int bn = conv_halo_bn(ncol);
  const int64_t bands = ((int64_t)a.nx * a.H + TR - 1) / TR;
  const int zb = (ncol + bn - 1) / bn;
  if ((bands + 7) / 8 * 8 * zb >= (1 << 30)) return hipErrorInvalidValue;
  a.bands = (int)bands;
  a.zblocks = zb;
  dim3 grid((unsigned)((bands + 7) / 8 * 8 * zb), (unsigned)nslots, 1);
  switch (a.W) {
    case 8: return launch_halo_w<8>(a, grid, bn, s);
    case 16: return launch_halo_w<16>(a, grid, bn, s);
    case 32: return launch_halo_w<32>(a, grid, bn, s);
    default: return launch_halo_w<64>(a, grid, bn, s);
  }
}

}  // namespace mure
