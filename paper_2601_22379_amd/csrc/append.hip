// Append path: key/value rows into the cache, block key statistics, and the
// global linear-attention state S_bar = sum_t phi(k_t)^T v_t, z_bar =
// sum_t phi(k_t) (Sec. 3.1 statistics, Sec. 3.2 Eq. 15, phi = softmax over
// the feature dimension).
#include "spla_device.h"
#include "spla_kernels.h"

namespace spla {

// Tokens of sequence b this append really adds (clamped to the capacity).
__device__ __forceinline__ int appended_count(const Dims& m, int L0, int max_new,
                                              const int32_t* __restrict__ n_new, int b,
                                              bool* clipped) {
  int n = n_new ? n_new[b] : max_new;
  n = n < 0 ? 0 : (n > max_new ? max_new : n);
  int room = m.cap - L0;
  room = room < 0 ? 0 : room;
  *clipped = n > room;
  return n < room ? n : room;
}

// One workgroup per touched statistics unit (a block, or a strided selection
// window: unit u holds tokens u us .. u us + ul - 1): merges the new tokens
// of the unit into its statistics and copies the rows t with
// u us <= t < (u + 1) us into the caches, so that each row is copied by
// exactly one unit. The new tokens' mean and M2 are computed two-pass in fp64
// and combined with the stored ones by Chan's formula, then rounded to fp32.
// (unit ux of the units touched, of (sequence, kv head) bh; thread j handles
// coordinate j). New row r of bh is element bh * s_bh + r * s_row of k_new
// and v_new: s_bh = max_new d, s_row = d for [batch][Hkv][max_new][d]
// (spla_append), s_bh = d, s_row = batch Hkv d for position-major rows
// [max_new][batch][Hkv][d] (the chunked prefill).
template <typename T>
__device__ __forceinline__ void append_unit(
    const Dims& m, T* __restrict__ kc, T* __restrict__ vc, float* __restrict__ stats,
    const int32_t* __restrict__ seq_lens, int32_t* __restrict__ err, const T* __restrict__ k_new,
    const T* __restrict__ v_new, int max_new, const int32_t* __restrict__ n_new,
    const int32_t* __restrict__ table, int ux, int bh, int64_t s_bh, int64_t s_row) {
  const int b = bh / m.hkv;
  const int L0 = seq_lens[b];
  bool clipped;
  const int ne = appended_count(m, L0, max_new, n_new, b, &clipped);
  if (clipped && err && ux == 0 && bh % m.hkv == 0 && threadIdx.x == 0)
    atomicOr(err, (int)SPLA_DEVERR_CAPACITY);
  // first unit holding token L0: u us + ul > L0
  const int first = L0 >= m.ul ? (L0 - m.ul) / m.us + 1 : 0;
  const int i = first + ux;
  const int t_lo = max(L0, i * m.us);
  const int t_hi = min(L0 + ne, i * m.us + m.ul);
  const int t_own = min(t_hi, (i + 1) * m.us);  // rows this unit copies: t_lo .. t_own - 1
  const int j = threadIdx.x;
  if (t_hi <= t_lo || j >= m.d) return;
  const int64_t src0 = (int64_t)bh * s_bh - (int64_t)L0 * s_row + j;  // row t at src0 + t s_row

  // the slot of the block that holds the rows this unit copies (they all lie
  // in one block: a unit's first us tokens, us dividing B); -1: a paged
  // table entry out of range, the rows are not written
  int64_t slot = -1;
  if (t_own > t_lo) {
    const int blk = t_lo / m.B;
    if (!table) {
      slot = (int64_t)bh * m.nb_cap + blk;
    } else {
      const int p = block_page(m, table, bh, blk);
      slot = p < 0 ? -1 : (int64_t)p * m.hkv + bh % m.hkv;
      if (p < 0 && err && j == 0) atomicOr(err, (int)SPLA_DEVERR_PAGE);
    }
  }
  double sum = 0.0;
  for (int t = t_lo; t < t_hi; ++t) {
    const T kv = k_new[src0 + (int64_t)t * s_row];
    if (t < t_own && slot >= 0) {
      kc[k_off_slot(m, slot, t % m.B, j)] = kv;
      vc[v_off_slot(m, slot, t % m.B, j)] = v_new[src0 + (int64_t)t * s_row];
    }
    sum += (double)Elem<T>::load(&kv, 0);
  }
  const int nc = t_hi - t_lo;
  const double mean_c = sum / nc;
  double m2_c = 0.0;
  for (int t = t_lo; t < t_hi; ++t) {
    const double x = (double)Elem<T>::load(k_new, src0 + (int64_t)t * s_row) - mean_c;
    m2_c += x * x;
  }
  const int na = t_lo - i * m.us;
  const int64_t o_mean = stats_off4(m, bh, i, 0, j / 4) + (j & 3);
  const int64_t o_m2 = stats_off4(m, bh, i, 1, j / 4) + (j & 3);
  double mean = mean_c, m2 = m2_c;
  if (na > 0) {
    const double mean_a = stats[o_mean], m2_a = stats[o_m2];
    const double n = (double)(na + nc);
    const double delta = mean_c - mean_a;
    mean = mean_a + delta * (nc / n);
    m2 = m2_a + m2_c + delta * delta * ((double)na * nc / n);
  }
  stats[o_mean] = (float)mean;
  stats[o_m2] = (float)m2;
}

// Bulk form of append_unit: 256 threads per unit. Thread (token lane tl,
// coordinate group cq) moves VEC = 16 / element-size coordinates of a row as
// one 16-byte access; with NQ = d / VEC groups there are TS = 256 / NQ token
// lanes, and lane tl takes the unit's tokens tl, tl + TS, ... . Key rows go
// to the cache as they are (a 16-byte piece of a row is one piece of the
// cache layout); value rows are staged in LDS and written out as the pieces
// of the cache layout (8 tokens of one coordinate for bf16, 4 for fp32);
// pieces not wholly inside the rows this unit copies are written element by
// element. Statistics as in append_unit: two passes in fp64 over the new
// tokens (the token lanes' partial sums added in a fixed tree: first the
// lanes of a wavefront by lane swaps, then the four wavefronts), Chan's
// combination with the stored ones, rounded to fp32.
constexpr int kAppendUnitRows = 128;  // rows a unit copies at most (us <= B <= 128)

template <typename T>
__global__ __launch_bounds__(256) void append_blocks_kernel(
    Dims m, T* __restrict__ kc, T* __restrict__ vc, float* __restrict__ stats,
    const int32_t* __restrict__ seq_lens, int32_t* __restrict__ err, const T* __restrict__ k_new,
    const T* __restrict__ v_new, int max_new, const int32_t* __restrict__ n_new,
    const int32_t* __restrict__ table, int64_t s_bh, int64_t s_row) {
  constexpr int VEC = 16 / (int)sizeof(T);
  __shared__ double part[4 * 128];  // per wavefront and coordinate
  __shared__ double smean[128];
  __shared__ __align__(16) T sV[kAppendUnitRows * 128];
  const int ux = (int)blockIdx.x, bh = (int)blockIdx.y;
  const int b = bh / m.hkv;
  const int L0 = seq_lens[b];
  bool clipped;
  const int ne = appended_count(m, L0, max_new, n_new, b, &clipped);
  if (clipped && err && ux == 0 && bh % m.hkv == 0 && threadIdx.x == 0)
    atomicOr(err, (int)SPLA_DEVERR_CAPACITY);
  const int first = L0 >= m.ul ? (L0 - m.ul) / m.us + 1 : 0;
  const int i = first + ux;
  const int t_lo = max(L0, i * m.us);
  const int t_hi = min(L0 + ne, i * m.us + m.ul);
  const int t_own = min(t_hi, (i + 1) * m.us);  // rows this unit copies: t_lo .. t_own - 1
  if (t_hi <= t_lo) return;  // uniform over the workgroup
  const int d = m.d, NQ = d / VEC, TS = 256 / NQ;
  const int tid = (int)threadIdx.x, cq = tid % NQ, tl = tid / NQ, c0 = cq * VEC;
  const int64_t src0 = (int64_t)bh * s_bh - (int64_t)L0 * s_row + c0;  // row t at src0 + t s_row
  int64_t slot = -1;
  if (t_own > t_lo) {
    const int blk = t_lo / m.B;
    if (!table) {
      slot = (int64_t)bh * m.nb_cap + blk;
    } else {
      const int p = block_page(m, table, bh, blk);
      slot = p < 0 ? -1 : (int64_t)p * m.hkv + bh % m.hkv;
      if (p < 0 && err && tid == 0) atomicOr(err, (int)SPLA_DEVERR_PAGE);
    }
  }
  // pass 1: key rows to the cache, value rows to LDS, sums of the keys
  double sum[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) sum[e] = 0.0;
  for (int t0 = t_lo + tl; t0 < t_hi; t0 += TS * 4) {
    uint4 kv[4], vv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int t = min(t0 + u * TS, t_hi - 1);
      kv[u] = *reinterpret_cast<const uint4*>(k_new + src0 + (int64_t)t * s_row);
      vv[u] = *reinterpret_cast<const uint4*>(v_new + src0 + (int64_t)t * s_row);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int t = t0 + u * TS;
      if (t < t_hi) {
        if (t < t_own && slot >= 0) {
          *reinterpret_cast<uint4*>(kc + k_off_slot(m, slot, t % m.B, c0)) = kv[u];
          *reinterpret_cast<uint4*>(sV + (t - t_lo) * d + c0) = vv[u];
        }
        const T* x = reinterpret_cast<const T*>(&kv[u]);
#pragma unroll
        for (int e = 0; e < VEC; ++e) sum[e] += (double)Elem<T>::load(x, e);
      }
    }
  }
  // the token lanes of this wavefront (lanes cq, cq + NQ, ...), then one
  // entry per wavefront and coordinate
  const int w = tid >> 6, lane = tid & 63;
  auto lanes_sum = [&](double (&v)[VEC]) {
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      for (int sft = NQ; sft < 64; sft *= 2) v[e] += __shfl_xor(v[e], sft, 64);
      if (lane < NQ) part[w * d + c0 + e] = v[e];
    }
  };
  lanes_sum(sum);
  __syncthreads();
  // value pieces: PV tokens of one coordinate each
  if (slot >= 0) {
    constexpr int PV = VEC;
    const int g_lo = t_lo - t_lo % PV;
    const int n_pieces = ((t_own + PV - 1) / PV - g_lo / PV) * d;
    for (int pc = tid; pc < n_pieces; pc += 256) {
      const int c = pc % d, tg = g_lo + (pc / d) * PV;  // first token of the piece
      if (tg >= t_lo && tg + PV <= t_own) {
        T x[PV];
#pragma unroll
        for (int e = 0; e < PV; ++e) x[e] = sV[(tg + e - t_lo) * d + c];
        *reinterpret_cast<uint4*>(vc + v_off_slot(m, slot, tg % m.B, c)) =
            *reinterpret_cast<const uint4*>(x);
      } else {
        for (int e = 0; e < PV; ++e) {
          const int t = tg + e;
          if (t >= t_lo && t < t_own) vc[v_off_slot(m, slot, t % m.B, c)] = sV[(t - t_lo) * d + c];
        }
      }
    }
  }
  const int nc = t_hi - t_lo;
  double mean_c[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) {
    const int c = c0 + e;
    mean_c[e] = (((part[c] + part[d + c]) + part[2 * d + c]) + part[3 * d + c]) / nc;
    if (tl == 0) smean[c] = mean_c[e];
  }
  __syncthreads();
  // pass 2: sum of squared deviations from the new tokens' mean
  double m2[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) m2[e] = 0.0;
  for (int t0 = t_lo + tl; t0 < t_hi; t0 += TS * 4) {
    uint4 kv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
      kv[u] = *reinterpret_cast<const uint4*>(k_new + src0 +
                                              (int64_t)min(t0 + u * TS, t_hi - 1) * s_row);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const T* x = reinterpret_cast<const T*>(&kv[u]);
      const bool ok = t0 + u * TS < t_hi;
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const double dx = (double)Elem<T>::load(x, e) - mean_c[e];
        m2[e] += ok ? dx * dx : 0.0;
      }
    }
  }
  lanes_sum(m2);
  __syncthreads();
  // coordinate j = tid (d threads): combine with the stored statistics
  if (tid >= d) return;
  const int j = tid;
  const double m2s = ((part[j] + part[d + j]) + part[2 * d + j]) + part[3 * d + j];
  const double mc = smean[j];
  const int na = t_lo - i * m.us;
  const int64_t o_mean = stats_off4(m, bh, i, 0, j / 4) + (j & 3);
  const int64_t o_m2 = stats_off4(m, bh, i, 1, j / 4) + (j & 3);
  double mean = mc, m2v = m2s;
  if (na > 0) {
    const double mean_a = stats[o_mean], m2_a = stats[o_m2];
    const double n = (double)(na + nc);
    const double delta = mc - mean_a;
    mean = mean_a + delta * (nc / n);
    m2v = m2_a + m2s + delta * delta * ((double)na * nc / n);
  }
  stats[o_mean] = (float)mean;
  stats[o_m2] = (float)m2v;
}

// Partial linear-attention state of one chunk of new tokens:
// P[j][c] = sum_t phi(k_t)_j v_t,c and Pz[j] = sum_t phi(k_t)_j, fp32.
template <typename T, int D>
__global__ __launch_bounds__(256) void append_state_partial_kernel(
    Dims m, const int32_t* __restrict__ seq_lens, const T* __restrict__ k_new,
    const T* __restrict__ v_new, int max_new, const int32_t* __restrict__ n_new, int n_chunks,
    int chunk_tokens, float* __restrict__ part_s, float* __restrict__ part_z) {
  constexpr int R = D / 16;
  __shared__ float sE[kSubTokens][D + 1];
  __shared__ float sV[kSubTokens][D + 1];
  const int bh = blockIdx.y;
  const int b = bh / m.hkv;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  bool clipped;
  const int ne = appended_count(m, seq_lens[b], max_new, n_new, b, &clipped);
  const int t0 = blockIdx.x * chunk_tokens;
  const int t1 = min(t0 + chunk_tokens, ne);
  const int tr = tid / 16, tc = tid % 16;
  float acc[R][R];
  float zacc[R];
#pragma unroll
  for (int a = 0; a < R; ++a) {
    zacc[a] = 0.f;
#pragma unroll
    for (int c = 0; c < R; ++c) acc[a][c] = 0.f;
  }
  for (int tt = t0; tt < t1; tt += kSubTokens) {
    const int nt = min(kSubTokens, t1 - tt);
    for (int e = tid; e < kSubTokens * D; e += 256) {
      const int row = e / D, col = e % D;
      const int64_t src = ((int64_t)bh * max_new + tt + row) * D + col;
      sE[row][col] = row < nt ? Elem<T>::load(k_new, src) : 0.f;
      sV[row][col] = row < nt ? Elem<T>::load(v_new, src) : 0.f;
    }
    __syncthreads();
    // phi(k) = softmax over the feature dimension, one row per wave step
    for (int r = 0; r < kSubTokens / 4; ++r) {
      const int row = w * (kSubTokens / 4) + r;
      float x[D / 64];
      float mx = -INFINITY;
#pragma unroll
      for (int e = 0; e < D / 64; ++e) {
        x[e] = sE[row][lane + 64 * e];
        mx = fmaxf(mx, x[e]);
      }
      mx = wave_max(mx);
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < D / 64; ++e) {
        x[e] = expf(x[e] - mx);
        s += x[e];
      }
      s = wave_sum(s);
      const float inv = row < nt ? 1.0f / s : 0.f;
#pragma unroll
      for (int e = 0; e < D / 64; ++e) sE[row][lane + 64 * e] = x[e] * inv;
    }
    __syncthreads();
    for (int t = 0; t < nt; ++t) {
      float pv[R], vv[R];
#pragma unroll
      for (int a = 0; a < R; ++a) {
        pv[a] = sE[t][tr * R + a];
        vv[a] = sV[t][tc * R + a];
      }
#pragma unroll
      for (int a = 0; a < R; ++a) {
        zacc[a] += pv[a];
#pragma unroll
        for (int c = 0; c < R; ++c) acc[a][c] = fmaf(pv[a], vv[c], acc[a][c]);
      }
    }
    __syncthreads();
  }
  float* ps = part_s + ((int64_t)bh * n_chunks + blockIdx.x) * D * D;
#pragma unroll
  for (int a = 0; a < R; ++a)
#pragma unroll
    for (int c = 0; c < R; ++c) ps[(tr * R + a) * D + tc * R + c] = acc[a][c];
  if (tc == 0) {
    float* pz = part_z + ((int64_t)bh * n_chunks + blockIdx.x) * D;
#pragma unroll
    for (int a = 0; a < R; ++a) pz[tr * R + a] = zacc[a];
  }
}

// The same partial state on the matrix cores (bf16 keys and values), one
// workgroup per (chunk, sequence x KV head). Per 32-token step, phi(k) of the
// step's keys (softmax over d, fp32) goes to LDS transposed as bf16 hi + lo
// (the A operand, rows = coordinates j, k = tokens), the values transposed
// (the B operand, columns = coordinates c); then
//   P[j][c] += sum_t phi(k_t)_j v_t,c
// on v_mfma_f32_16x16x32_bf16 (hi and lo products, fp32 accumulation).
// Wavefront w owns columns (D / 4) w .. of P: D / 16 row tiles x D / 64
// column tiles. Each wavefront reads its 8 tokens of a step with 16-byte
// loads, D / 8 lanes per token, and takes the softmax's max and sum over a
// token's lanes by DPP (two-byte loads, one token at a time with full-wave
// reductions, took 146 us for a 16K-token slab at 128K). Pz accumulates
// phi(k) in fp32 per lane.
typedef __bf16 abf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 abf16x2 __attribute__((ext_vector_type(2)));
typedef float afloatx2 __attribute__((ext_vector_type(2)));

// Two floats rounded to bf16 (nearest even) by one packed conversion: a in
// the low half, b in the high half.
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(afloatx2{a, b}, abf16x2));
}
typedef float afloatx4 __attribute__((ext_vector_type(4)));

// Coordinate c's row of a transposed array starts at c TPP + 8 (c / 8): the
// pad after every 8 rows puts the 16 coordinate groups a wavefront writes at
// once (one token of 8 coordinates per lane) on 16 different banks, and
// keeps every row 16-byte aligned for the operand reads.
template <int D>
struct alignas(16) StateSmem {
  static constexpr int TPP = kSubTokens + 8;
  static constexpr int N = D * TPP + D;
  static __device__ __forceinline__ int at(int c, int t) { return c * TPP + 8 * (c >> 3) + t; }
  uint16_t kT_h[N], kT_l[N];  // phi(k)^T of the step
  uint16_t vT[N];             // v^T of the step
  float z[4][D];              // per-wavefront sums of phi(k)
};

template <int D>
__global__ __launch_bounds__(256) void append_state_mfma_kernel(
    Dims m, const int32_t* __restrict__ seq_lens, const bf16_t* __restrict__ k_new,
    const bf16_t* __restrict__ v_new, int max_new, const int32_t* __restrict__ n_new, int n_chunks,
    int chunk_tokens, float* __restrict__ part_s, float* __restrict__ part_z) {
  constexpr int RT = D / 16;        // row tiles (coordinates j)
  constexpr int CT = D / 64;        // column tiles per wavefront
  __shared__ StateSmem<D> sm;
  const int bh = blockIdx.y;
  const int b = bh / m.hkv;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int li = lane & 15, lg = lane >> 4;
  bool clipped;
  const int ne = appended_count(m, seq_lens[b], max_new, n_new, b, &clipped);
  const int t0 = blockIdx.x * chunk_tokens;
  const int t1 = min(t0 + chunk_tokens, ne);
  afloatx4 acc[RT][CT];
#pragma unroll
  for (int r = 0; r < RT; ++r)
#pragma unroll
    for (int c = 0; c < CT; ++c) acc[r][c] = afloatx4{0.f, 0.f, 0.f, 0.f};
  float zacc[8];  // phi(k) of this lane's coordinates, summed over its tokens
#pragma unroll
  for (int i = 0; i < 8; ++i) zacc[i] = 0.f;
  const bf16_t* kb = k_new + (int64_t)bh * max_new * D;
  const bf16_t* vb = v_new + (int64_t)bh * max_new * D;
  // wavefront w takes tokens 8 w .. 8 w + 7 of each 32-token step as NS
  // 16-byte loads per lane: LPR = D / 8 lanes per token, lane l holding
  // coordinates 8 (l % LPR) .. + 7 of token tok(s) (with two loads, tokens
  // 2 tl and 2 tl + 1, tl = l / LPR: the lane then writes both tokens of a
  // coordinate to the transposed arrays as one 4-byte store); the next
  // step's rows are loaded while the current one is processed
  constexpr int LPR = D / 8, RPL = 64 / LPR, NS = 8 / RPL;
  const int cl = lane % LPR, tl = lane / LPR;
  auto tok = [&](int s) { return 8 * w + (NS == 2 ? 2 * tl + s : RPL * s + tl); };
  uint4 kx[NS], vx[NS];
  auto load_step = [&](int tt) {
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const int row = min(tt + tok(s), t1 - 1);
      kx[s] = *reinterpret_cast<const uint4*>(kb + (int64_t)row * D + 8 * cl);
      vx[s] = *reinterpret_cast<const uint4*>(vb + (int64_t)row * D + 8 * cl);
    }
  };
  // max / sum over the LPR lanes of a token (every lane gets the same bits)
  auto row_max = [](float v) {
    if constexpr (LPR == 16) {
      v = fmaxf(v, dpp_rot<0x128>(v));  // row_ror:8
      v = fmaxf(v, dpp_rot<0x124>(v));  // row_ror:4
    } else {
      v = fmaxf(v, dpp_rot<0x141>(v));  // row_half_mirror
    }
    v = fmaxf(v, dpp_rot<0x4E>(v));
    return fmaxf(v, dpp_rot<0xB1>(v));
  };
  auto row_sum = [](float v) {
    if constexpr (LPR == 16) {
      v += dpp_rot<0x128>(v);
      v += dpp_rot<0x124>(v);
    } else {
      v += dpp_rot<0x141>(v);
    }
    v += dpp_rot<0x4E>(v);
    return v + dpp_rot<0xB1>(v);
  };
  if (t0 < t1) load_step(t0);
  for (int tt = t0; tt < t1; tt += kSubTokens) {
    const int nt = min(kSubTokens, t1 - tt);
    uint4 kc[NS], vc[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      kc[s] = kx[s];
      vc[s] = vx[s];
    }
    if (tt + kSubTokens < t1) load_step(tt + kSubTokens);
    float ph[NS][8];  // phi(k) of the token of load s, coordinates 8 cl + i
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const bool ok = tok(s) < nt;
      const uint32_t kw[4] = {kc[s].x, kc[s].y, kc[s].z, kc[s].w};
      float kf[8];
#pragma unroll
      for (int i = 0; i < 8; ++i)
        kf[i] = bf16_to_f32((uint16_t)(i & 1 ? kw[i >> 1] >> 16 : kw[i >> 1] & 0xFFFFu));
      float mx = kf[0];
#pragma unroll
      for (int i = 1; i < 8; ++i) mx = fmaxf(mx, kf[i]);
      mx = row_max(mx);
      // exp(k - max k) as the sparse pass forms it (hardware exp2); the sum
      // is in [1, D], where the hardware reciprocal is within 1 ulp
      const float mxl = mx * kLog2e;
      float sum = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        kf[i] = __builtin_amdgcn_exp2f(fmaf(kf[i], kLog2e, -mxl));
        sum += kf[i];
      }
      sum = row_sum(sum);
      const float inv = ok ? __builtin_amdgcn_rcpf(sum) : 0.f;  // phi = 0 past the chunk
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        ph[s][i] = kf[i] * inv;
        zacc[i] += ph[s][i];
      }
    }
    if constexpr (NS == 2) {
      // tokens 2 tl, 2 tl + 1 of coordinate 8 cl + i as one 4-byte store
      // each: hi pair rounded by one packed conversion, lo = phi - hi; the
      // value pair by one byte permute (rows past the chunk hold real,
      // finite values and meet phi = 0)
      const uint32_t v0[4] = {vc[0].x, vc[0].y, vc[0].z, vc[0].w};
      const uint32_t v1[4] = {vc[1].x, vc[1].y, vc[1].z, vc[1].w};
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t hp = pack_bf16x2(ph[0][i], ph[1][i]);
        const float h0 = __uint_as_float(hp << 16), h1 = __uint_as_float(hp & 0xFFFF0000u);
        const uint32_t lp = pack_bf16x2(ph[0][i] - h0, ph[1][i] - h1);
        const uint32_t vp =
            __builtin_amdgcn_perm(v1[i >> 1], v0[i >> 1], i & 1 ? 0x07060302u : 0x05040100u);
        const int o = StateSmem<D>::at(8 * cl + i, tok(0));
        *reinterpret_cast<uint32_t*>(&sm.kT_h[o]) = hp;
        *reinterpret_cast<uint32_t*>(&sm.kT_l[o]) = lp;
        *reinterpret_cast<uint32_t*>(&sm.vT[o]) = vp;
      }
    } else {
      const uint32_t vw[4] = {vc[0].x, vc[0].y, vc[0].z, vc[0].w};
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const __bf16 hi = (__bf16)ph[0][i];
        const __bf16 lo = (__bf16)(ph[0][i] - (float)hi);
        const int o = StateSmem<D>::at(8 * cl + i, tok(0));
        sm.kT_h[o] = __builtin_bit_cast(uint16_t, hi);
        sm.kT_l[o] = __builtin_bit_cast(uint16_t, lo);
        sm.vT[o] = (uint16_t)(i & 1 ? vw[i >> 1] >> 16 : vw[i >> 1] & 0xFFFFu);
      }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      const int oa = StateSmem<D>::at(16 * r + li, 8 * lg);
      const abf16x8 ah =
          __builtin_bit_cast(abf16x8, *reinterpret_cast<const uint4*>(&sm.kT_h[oa]));
      const abf16x8 al =
          __builtin_bit_cast(abf16x8, *reinterpret_cast<const uint4*>(&sm.kT_l[oa]));
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        const int col = (D / 4) * w + 16 * c + li;
        const abf16x8 bv = __builtin_bit_cast(
            abf16x8, *reinterpret_cast<const uint4*>(&sm.vT[StateSmem<D>::at(col, 8 * lg)]));
        acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bv, acc[r][c], 0, 0, 0);
        acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bv, acc[r][c], 0, 0, 0);
      }
    }
    __syncthreads();
  }
  float* ps = part_s + ((int64_t)bh * n_chunks + blockIdx.x) * D * D;
#pragma unroll
  for (int r = 0; r < RT; ++r)
#pragma unroll
    for (int c = 0; c < CT; ++c)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4)
        ps[(16 * r + 4 * lg + r4) * D + (D / 4) * w + 16 * c + li] = acc[r][c][r4];
  // the lanes of one coordinate group: l, l + LPR, ... (LPR = 16: xor 16,
  // xor 32; LPR = 8: first the other half of the 16-lane row)
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float v = zacc[i];
    if constexpr (LPR == 8) v += dpp_rot<0x128>(v);
    v += xor16(v);
    v += xor32(v);
    zacc[i] = v;
  }
  if (lane < LPR) {
#pragma unroll
    for (int i = 0; i < 8; ++i) sm.z[w][8 * lane + i] = zacc[i];
  }
  __syncthreads();
  if (tid < D) {
    float z = 0.f;
#pragma unroll
    for (int x = 0; x < 4; ++x) z += sm.z[x][tid];
    part_z[((int64_t)bh * n_chunks + blockIdx.x) * D + tid] = z;
  }
}

// Bulk append in one pass over the new keys and values (bf16, d = 128, one
// statistics unit per block): one workgroup per (chunk, sequence x KV head),
// the chunks aligned to blocks (chunk x covers positions a0 .. a0 + ct - 1,
// a0 = L0 - L0 % B + x ct), so that every block's statistics belong to one
// workgroup. Per 32-token step (one block holds whole steps) the workgroup
//   * writes the step's key rows to the cache from the registers they were
//     loaded into (a 16-byte piece of a row is one piece of the cache);
//   * leaves phi(k) (bf16 hi + lo), the values and the keys transposed in
//     LDS, and adds the step to the chunk's partial state on the matrix
//     cores (as append_state_mfma_kernel, bit for bit);
//   * writes the value pieces of the cache (8 tokens of one coordinate)
//     from the transposed values;
//   * adds the step's keys to the block's sums of k and k^2 per coordinate
//     in fp64 (two threads per coordinate, 16 tokens each: exact for bf16
//     keys over a block), and after the block's last step merges the new
//     tokens' mean and M2 = sum k^2 - mean sum k into the stored statistics
//     (Chan's combination, rounded to fp32).
// Tokens outside [L0, L0 + n) (before the append point in the first block,
// past the new tokens in the last) load a clamped real row, get phi = 0 and
// are neither stored nor counted.
template <int D>
__global__ __launch_bounds__(256) void append_fused_kernel(
    Dims m, bf16_t* __restrict__ kcache, bf16_t* __restrict__ vcache, float* __restrict__ stats,
    const int32_t* __restrict__ seq_lens, int32_t* __restrict__ err,
    const bf16_t* __restrict__ k_new, const bf16_t* __restrict__ v_new, int max_new,
    const int32_t* __restrict__ n_new, const int32_t* __restrict__ table, int n_chunks,
    int chunk_tokens, float* __restrict__ part_s, float* __restrict__ part_z) {
  static_assert(D == 128, "two tokens per lane: d = 128");
  constexpr int RT = D / 16;  // row tiles (coordinates j)
  constexpr int CT = D / 64;  // column tiles per wavefront
  __shared__ StateSmem<D> sm;
  __shared__ __align__(16) uint16_t kR[StateSmem<D>::N];  // keys of the step, transposed
  const int bh = blockIdx.y;
  const int b = bh / m.hkv;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int li = lane & 15, lg = lane >> 4;
  const int L0 = seq_lens[b];
  bool clipped;
  const int ne = appended_count(m, L0, max_new, n_new, b, &clipped);
  if (clipped && err && blockIdx.x == 0 && bh % m.hkv == 0 && tid == 0)
    atomicOr(err, (int)SPLA_DEVERR_CAPACITY);
  const int Bk = m.B;
  const int a0 = L0 - L0 % Bk + (int)blockIdx.x * chunk_tokens;
  const int lo = max(a0, L0), a1n = min(a0 + chunk_tokens, L0 + ne);
  const int a1 = lo < a1n ? a1n : a0;  // no step when the chunk holds no new token
  afloatx4 acc[RT][CT];
#pragma unroll
  for (int r = 0; r < RT; ++r)
#pragma unroll
    for (int c = 0; c < CT; ++c) acc[r][c] = afloatx4{0.f, 0.f, 0.f, 0.f};
  float zacc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) zacc[i] = 0.f;
  const bf16_t* kb = k_new + (int64_t)bh * max_new * D;
  const bf16_t* vb = v_new + (int64_t)bh * max_new * D;
  // lane l: coordinates 8 (l % 16) .. + 7 of tokens 8 w + 2 (l / 16) + s
  const int cl = lane & 15, tl = lane >> 4;
  auto tok = [&](int s) { return 8 * w + 2 * tl + s; };
  uint4 kx[2], vx[2];
  auto load_step = [&](int tt) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int row = min(max(tt + tok(s) - L0, 0), ne - 1);
      kx[s] = *reinterpret_cast<const uint4*>(kb + (int64_t)row * D + 8 * cl);
      vx[s] = *reinterpret_cast<const uint4*>(vb + (int64_t)row * D + 8 * cl);
    }
  };
  auto row_max = [](float v) {
    v = fmaxf(v, dpp_rot<0x128>(v));  // row_ror:8
    v = fmaxf(v, dpp_rot<0x124>(v));  // row_ror:4
    v = fmaxf(v, dpp_rot<0x4E>(v));
    return fmaxf(v, dpp_rot<0xB1>(v));
  };
  auto row_sum = [](float v) {
    v += dpp_rot<0x128>(v);
    v += dpp_rot<0x124>(v);
    v += dpp_rot<0x4E>(v);
    return v + dpp_rot<0xB1>(v);
  };
  // statistics: thread (coordinate sc, half sh) sums tokens 16 sh .. + 15
  const int sc = tid >> 1, sh = tid & 1;
  double s1 = 0.0, s2 = 0.0;
  int64_t slot = -1;
  if (a0 < a1) load_step(a0);
  for (int tt = a0; tt < a1; tt += kSubTokens) {
    const int blk = tt / Bk;
    if (tt % Bk == 0) {  // a block starts: its slot in the caches
      if (!table) {
        slot = (int64_t)bh * m.nb_cap + blk;
      } else {
        const int p = block_page(m, table, bh, blk);
        slot = p < 0 ? -1 : (int64_t)p * m.hkv + bh % m.hkv;
        if (p < 0 && err && tid == 0) atomicOr(err, (int)SPLA_DEVERR_PAGE);
      }
    }
    uint4 kc[2], vc[2];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      kc[s] = kx[s];
      vc[s] = vx[s];
    }
    if (tt + kSubTokens < a1) load_step(tt + kSubTokens);
    float ph[2][8];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int t = tt + tok(s);
      const bool ok = t >= lo && t < a1;
      if (ok && slot >= 0)
        *reinterpret_cast<uint4*>(kcache + k_off_slot(m, slot, t % Bk, 8 * cl)) = kc[s];
      const uint32_t kw[4] = {kc[s].x, kc[s].y, kc[s].z, kc[s].w};
      float kf[8];
#pragma unroll
      for (int i = 0; i < 8; ++i)
        kf[i] = bf16_to_f32((uint16_t)(i & 1 ? kw[i >> 1] >> 16 : kw[i >> 1] & 0xFFFFu));
      float mx = kf[0];
#pragma unroll
      for (int i = 1; i < 8; ++i) mx = fmaxf(mx, kf[i]);
      mx = row_max(mx);
      const float mxl = mx * kLog2e;
      float sum = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        kf[i] = __builtin_amdgcn_exp2f(fmaf(kf[i], kLog2e, -mxl));
        sum += kf[i];
      }
      sum = row_sum(sum);
      const float inv = ok ? __builtin_amdgcn_rcpf(sum) : 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        ph[s][i] = kf[i] * inv;
        zacc[i] += ph[s][i];
      }
    }
    {
      const uint32_t k0[4] = {kc[0].x, kc[0].y, kc[0].z, kc[0].w};
      const uint32_t k1[4] = {kc[1].x, kc[1].y, kc[1].z, kc[1].w};
      const uint32_t v0[4] = {vc[0].x, vc[0].y, vc[0].z, vc[0].w};
      const uint32_t v1[4] = {vc[1].x, vc[1].y, vc[1].z, vc[1].w};
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t sel = i & 1 ? 0x07060302u : 0x05040100u;
        const uint32_t hp = pack_bf16x2(ph[0][i], ph[1][i]);
        const float h0 = __uint_as_float(hp << 16), h1 = __uint_as_float(hp & 0xFFFF0000u);
        const int o = StateSmem<D>::at(8 * cl + i, tok(0));
        *reinterpret_cast<uint32_t*>(&sm.kT_h[o]) = hp;
        *reinterpret_cast<uint32_t*>(&sm.kT_l[o]) = pack_bf16x2(ph[0][i] - h0, ph[1][i] - h1);
        *reinterpret_cast<uint32_t*>(&sm.vT[o]) = __builtin_amdgcn_perm(v1[i >> 1], v0[i >> 1], sel);
        *reinterpret_cast<uint32_t*>(&kR[o]) = __builtin_amdgcn_perm(k1[i >> 1], k0[i >> 1], sel);
      }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      const int oa = StateSmem<D>::at(16 * r + li, 8 * lg);
      const abf16x8 ah =
          __builtin_bit_cast(abf16x8, *reinterpret_cast<const uint4*>(&sm.kT_h[oa]));
      const abf16x8 al =
          __builtin_bit_cast(abf16x8, *reinterpret_cast<const uint4*>(&sm.kT_l[oa]));
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        const int col = (D / 4) * w + 16 * c + li;
        const abf16x8 bv = __builtin_bit_cast(
            abf16x8, *reinterpret_cast<const uint4*>(&sm.vT[StateSmem<D>::at(col, 8 * lg)]));
        acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bv, acc[r][c], 0, 0, 0);
        acc[r][c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bv, acc[r][c], 0, 0, 0);
      }
    }
    // value pieces: piece p = (c >> 4, token group g, c & 15), the order of
    // the cache within a step, so consecutive threads write consecutive
    // pieces
    const bool whole = tt >= lo && tt + kSubTokens <= a1;  // uniform
    if (slot >= 0) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int p = tid + 256 * u;
        const int c = ((p >> 6) << 4) + (p & 15), g = (p >> 4) & 3;
        const uint4 x = *reinterpret_cast<const uint4*>(&sm.vT[StateSmem<D>::at(c, 8 * g)]);
        const int tb = (tt + 8 * g) % Bk;
        if (whole) {
          *reinterpret_cast<uint4*>(vcache + v_off_slot(m, slot, tb, c)) = x;
        } else {
          const uint16_t* xe = reinterpret_cast<const uint16_t*>(&x);
          for (int e = 0; e < 8; ++e) {
            const int t = tt + 8 * g + e;
            if (t >= lo && t < a1)
              reinterpret_cast<uint16_t*>(vcache)[v_off_slot(m, slot, tb + e, c)] = xe[e];
          }
        }
      }
    }
    // the block's sums of k and k^2 (coordinate sc, tokens 16 sh .. + 15)
    {
      const int ob = StateSmem<D>::at(sc, 16 * sh);
      const uint4 r0 = *reinterpret_cast<const uint4*>(&kR[ob]);
      const uint4 r1 = *reinterpret_cast<const uint4*>(&kR[ob + 8]);
      const uint32_t kw[8] = {r0.x, r0.y, r0.z, r0.w, r1.x, r1.y, r1.z, r1.w};
      if (whole) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const double x =
              (double)bf16_to_f32((uint16_t)(e & 1 ? kw[e >> 1] >> 16 : kw[e >> 1] & 0xFFFFu));
          s1 += x;
          s2 = fma(x, x, s2);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int t = tt + 16 * sh + e;
          const double x =
              (t >= lo && t < a1)
                  ? (double)bf16_to_f32((uint16_t)(e & 1 ? kw[e >> 1] >> 16 : kw[e >> 1] & 0xFFFFu))
                  : 0.0;
          s1 += x;
          s2 = fma(x, x, s2);
        }
      }
    }
    if ((tt + kSubTokens) % Bk == 0 || tt + kSubTokens >= a1) {  // the block's last step
      s1 += __shfl_xor(s1, 1, 64);
      s2 += __shfl_xor(s2, 1, 64);
      if (sh == 0) {
        const int nc = min((blk + 1) * Bk, a1) - max(blk * Bk, lo);
        const int na = max(L0 - blk * Bk, 0);
        const double mc = s1 / nc;
        const double m2s = s2 - mc * s1;
        const int64_t o_mean = stats_off4(m, bh, blk, 0, sc / 4) + (sc & 3);
        const int64_t o_m2 = stats_off4(m, bh, blk, 1, sc / 4) + (sc & 3);
        double mean = mc, m2v = m2s;
        if (na > 0) {
          const double mean_a = stats[o_mean], m2_a = stats[o_m2];
          const double n = (double)(na + nc);
          const double delta = mc - mean_a;
          mean = mean_a + delta * (nc / n);
          m2v = m2_a + m2s + delta * delta * ((double)na * nc / n);
        }
        stats[o_mean] = (float)mean;
        stats[o_m2] = (float)m2v;
      }
      s1 = 0.0;
      s2 = 0.0;
    }
    __syncthreads();
  }
  float* ps = part_s + ((int64_t)bh * n_chunks + blockIdx.x) * D * D;
#pragma unroll
  for (int r = 0; r < RT; ++r)
#pragma unroll
    for (int c = 0; c < CT; ++c)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4)
        ps[(16 * r + 4 * lg + r4) * D + (D / 4) * w + 16 * c + li] = acc[r][c][r4];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    float v = zacc[i];
    v += xor16(v);
    v += xor32(v);
    zacc[i] = v;
  }
  if (lane < 16) {
#pragma unroll
    for (int i = 0; i < 8; ++i) sm.z[w][8 * lane + i] = zacc[i];
  }
  __syncthreads();
  if (tid < D) {
    float z = 0.f;
#pragma unroll
    for (int x = 0; x < 4; ++x) z += sm.z[x][tid];
    part_z[((int64_t)bh * n_chunks + blockIdx.x) * D + tid] = z;
  }
}

// S_bar += sum of the chunk partials, accumulated in fp64 in chunk order;
// kReduceRows rows of S_bar per workgroup (4: a thread has two entries at
// d = 128, and 32 x bh workgroups keep every compute unit busy).
constexpr int kReduceRows = 4;
// With seq_lens (the one-pass append), the first workgroup of each sequence
// also advances its length by the tokens appended (the append's last step:
// nothing in this kernel reads the lengths otherwise).
__global__ __launch_bounds__(256) void append_state_reduce_kernel(
    Dims m, int n_chunks, const float* __restrict__ part_s, const float* __restrict__ part_z,
    float* __restrict__ S, float* __restrict__ z, int32_t* __restrict__ seq_lens, int max_new,
    const int32_t* __restrict__ n_new) {
  const int bh = blockIdx.y;
  const int D = m.d;
  if (seq_lens && blockIdx.x == 0 && bh % m.hkv == 0 && threadIdx.x == 0) {
    const int b = bh / m.hkv;
    bool clipped;
    const int L0 = seq_lens[b];
    seq_lens[b] = L0 + appended_count(m, L0, max_new, n_new, b, &clipped);
  }
  const int row0 = blockIdx.x * kReduceRows;
  for (int e = threadIdx.x; e < kReduceRows * D; e += 256) {
    const int row = row0 + e / D, col = e % D;
    const int64_t o = ((int64_t)bh * D + row) * D + col;
    double s = S[o];
    const float* p = part_s + ((int64_t)bh * n_chunks * D + row) * D + col;  // chunk c at + c D D
    for (int c0 = 0; c0 < n_chunks; c0 += 16) {  // 16 loads in flight, added in chunk order
      float x[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) x[u] = p[(int64_t)min(c0 + u, n_chunks - 1) * D * D];
#pragma unroll
      for (int u = 0; u < 16; ++u) s += c0 + u < n_chunks ? (double)x[u] : 0.0;
    }
    S[o] = (float)s;
  }
  if (threadIdx.x < kReduceRows) {
    const int row = row0 + threadIdx.x;
    double s = z[(int64_t)bh * D + row];
    for (int c = 0; c < n_chunks; ++c) s += part_z[((int64_t)bh * n_chunks + c) * D + row];
    z[(int64_t)bh * D + row] = (float)s;
  }
}

// Single-token state update: S_bar += phi(k)^T v, z_bar += phi(k) (fp32).
// Rows rx * 16 .. rx * 16 + 15 of S_bar += phi(k)^T v (and those entries of
// z_bar += phi(k)) for the single token k, v of (sequence, kv head) bh, by the
// 256 threads of a workgroup. A sequence at capacity gets nothing.
template <typename T, int D>
__device__ __forceinline__ void append_rank1_rows(const Dims& m,
                                                  const int32_t* __restrict__ seq_lens,
                                                  const T* __restrict__ k_new,
                                                  const T* __restrict__ v_new,
                                                  float* __restrict__ S, float* __restrict__ z,
                                                  int rx, int bh) {
  __shared__ float sphi[D];
  __shared__ float sv[D];
  constexpr int PT = 16 * D / 256;  // entries of the 16 rows per thread
  const int b = bh / m.hkv;
  if (seq_lens[b] >= m.cap) return;
  const int tid = threadIdx.x;
  const int row0 = rx * 16;
  // this thread's entries of the rows, loaded before phi(k) is formed so that
  // their latency overlaps it
  float sr[PT];
#pragma unroll
  for (int u = 0; u < PT; ++u) {
    const int e = tid + 256 * u;
    sr[u] = S[((int64_t)bh * D + row0 + e / D) * D + e % D];
  }
  if (tid < 64) {
    float x[D / 64];
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < D / 64; ++e) {
      x[e] = Elem<T>::load(k_new, (int64_t)bh * D + tid + 64 * e);
      mx = fmaxf(mx, x[e]);
    }
    mx = wave_max(mx);
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < D / 64; ++e) {
      // exp(k - max k) as the sparse pass of this element type forms it
      x[e] = sizeof(T) == 2 ? __builtin_amdgcn_exp2f(fmaf(x[e], kLog2e, -mx * kLog2e))
                            : expf(x[e] - mx);
      s += x[e];
    }
    s = wave_sum(s);
#pragma unroll
    for (int e = 0; e < D / 64; ++e) sphi[tid + 64 * e] = x[e] / s;
  }
  for (int c = tid; c < D; c += 256) sv[c] = Elem<T>::load(v_new, (int64_t)bh * D + c);
  __syncthreads();
#pragma unroll
  for (int u = 0; u < PT; ++u) {
    const int e = tid + 256 * u;
    const int row = row0 + e / D, col = e % D;
    S[((int64_t)bh * D + row) * D + col] = fmaf(sphi[row], sv[col], sr[u]);
  }
  if (tid < 16) z[(int64_t)bh * D + row0 + tid] += sphi[row0 + tid];
}

// The end of a single-token append workgroup of (sequence, KV head) bh:
// the workgroups of a sequence (hkv x gridDim.x of them) count themselves in
// its counter (a line of the decode workspace's synchronisation area, zero
// between calls), and the last advances seq_lens[b] by the token appended (0
// at the capacity), writes that count to appended[b] (if not NULL) and
// resets the counter. Every workgroup has read seq_lens[b] before it counts
// itself, so no read of the old length follows the advance.
__device__ __forceinline__ void append_one_finish(const Dims& m, int32_t* seq_lens,
                                                  int32_t* fin_ctr, int32_t* appended, int bh,
                                                  int* s_flag) {
  const int b = bh / m.hkv;
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t* c = fin_ctr + (int64_t)b * kSyncLine;
    if (atomic_add_agent(c, 1) == m.hkv * (int)gridDim.x - 1) {
      bool clipped;
      const int L0 = seq_lens[b];
      const int n = appended_count(m, L0, 1, nullptr, b, &clipped);
      seq_lens[b] = L0 + n;
      if (appended) appended[b] = n;
      store_agent(c, 0);
    }
  }
}

// The single-token append of a decode step in one launch: workgroups
// x < D / 16 update 16 rows of S_bar each (rank one), the others the
// statistics units the token falls in (and copy its K/V rows). The two parts
// touch disjoint memory and only read seq_lens, which the last workgroup of
// each sequence advances afterwards (fin_ctr given: append_one_finish), or
// append_finish_kernel.
template <typename T, int D>
__global__ __launch_bounds__(256) void append_one_kernel(
    Dims m, T* __restrict__ kc, T* __restrict__ vc, float* __restrict__ stats,
    int32_t* __restrict__ seq_lens, int32_t* __restrict__ err, const T* __restrict__ k_new,
    const T* __restrict__ v_new, const int32_t* __restrict__ table, float* __restrict__ S,
    float* __restrict__ z, int32_t* __restrict__ fin_ctr, int32_t* __restrict__ appended) {
  __shared__ int s_flag;
  const int bh = (int)blockIdx.y;
  if ((int)blockIdx.x < D / 16)
    append_rank1_rows<T, D>(m, seq_lens, k_new, v_new, S, z, (int)blockIdx.x, bh);
  else
    append_unit<T>(m, kc, vc, stats, seq_lens, err, k_new, v_new, 1, nullptr, table,
                   (int)blockIdx.x - D / 16, bh, D, D);
  if (fin_ctr) append_one_finish(m, seq_lens, fin_ctr, appended, bh, &s_flag);
}

// The statistics units and K/V rows of a single-token append alone (the
// state's rank-one update is applied elsewhere): append_unit, d threads; then
// append_one_finish when fin_ctr is given.
template <typename T>
__global__ __launch_bounds__(128) void append_unit_kernel(
    Dims m, T* __restrict__ kc, T* __restrict__ vc, float* __restrict__ stats,
    int32_t* __restrict__ seq_lens, int32_t* __restrict__ err, const T* __restrict__ k_new,
    const T* __restrict__ v_new, const int32_t* __restrict__ table, int32_t* __restrict__ fin_ctr,
    int32_t* __restrict__ appended) {
  __shared__ int s_flag;
  append_unit<T>(m, kc, vc, stats, seq_lens, err, k_new, v_new, 1, nullptr, table,
                 (int)blockIdx.x, (int)blockIdx.y, m.d, m.d);
  if (fin_ctr) append_one_finish(m, seq_lens, fin_ctr, appended, (int)blockIdx.y, &s_flag);
}

// seq_lens[b] += the tokens appended; appended (if not NULL) receives that
// count per sequence.
__global__ void append_finish_kernel(Dims m, int32_t* __restrict__ seq_lens, int max_new,
                                     const int32_t* __restrict__ n_new,
                                     int32_t* __restrict__ appended) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= m.batch) return;
  bool clipped;
  const int L0 = seq_lens[b];
  const int n = appended_count(m, L0, max_new, n_new, b, &clipped);
  seq_lens[b] = L0 + n;
  if (appended) appended[b] = n;
}

__global__ void fill_zero_kernel(uint32_t* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

// ------------------------------------------------------------- launchers
hipError_t launch_append_blocks(const Dims& m, const spla_cache& c, const void* k_new,
                                const void* v_new, int max_new, const int32_t* n_new,
                                hipStream_t st, bool position_major) {
  // units touched by max_new tokens from any L0 (idle workgroups return)
  const int64_t nx = windowed(m) ? ceil_div(max_new + m.ul, m.us) + 2 : ceil_div(max_new, m.B) + 1;
  dim3 grid((unsigned)nx, (unsigned)m.bh);
  const int64_t s_bh = position_major ? m.d : (int64_t)max_new * m.d;
  const int64_t s_row = position_major ? (int64_t)m.bh * m.d : m.d;
  if (m.elem == 4)
    hipLaunchKernelGGL(append_blocks_kernel<float>, grid, dim3(256), 0, st, m, (float*)c.k_cache,
                       (float*)c.v_cache, c.blk_stats, c.seq_lens, c.err_flags,
                       (const float*)k_new, (const float*)v_new, max_new, n_new,
                       m.pages > 0 ? c.block_table : nullptr, s_bh, s_row);
  else
    hipLaunchKernelGGL(append_blocks_kernel<bf16_t>, grid, dim3(256), 0, st, m,
                       (bf16_t*)c.k_cache, (bf16_t*)c.v_cache, c.blk_stats, c.seq_lens,
                       c.err_flags, (const bf16_t*)k_new, (const bf16_t*)v_new, max_new, n_new,
                       m.pages > 0 ? c.block_table : nullptr, s_bh, s_row);
  return hipGetLastError();
}

template <typename T, int D>
static void state_partial(const Dims& m, const spla_cache& c, const void* k_new, const void* v_new,
                          int max_new, const int32_t* n_new, const AppendWs& ws, char* base,
                          hipStream_t st) {
  if constexpr (sizeof(T) == 2)
    hipLaunchKernelGGL((append_state_mfma_kernel<D>), dim3(ws.n_chunks, m.bh), dim3(256), 0, st,
                       m, c.seq_lens, (const bf16_t*)k_new, (const bf16_t*)v_new, max_new, n_new,
                       ws.n_chunks, ws.chunk_tokens, (float*)(base + ws.part_s),
                       (float*)(base + ws.part_z));
  else
    hipLaunchKernelGGL((append_state_partial_kernel<T, D>), dim3(ws.n_chunks, m.bh), dim3(256), 0,
                       st, m, c.seq_lens, (const T*)k_new, (const T*)v_new, max_new, n_new,
                       ws.n_chunks, ws.chunk_tokens, (float*)(base + ws.part_s),
                       (float*)(base + ws.part_z));
}

hipError_t launch_append_state(const Dims& m, const spla_cache& c, const void* k_new,
                               const void* v_new, int max_new, const int32_t* n_new,
                               const AppendWs& ws, char* base, hipStream_t st) {
  if (m.elem == 4) {
    if (m.d == 64) state_partial<float, 64>(m, c, k_new, v_new, max_new, n_new, ws, base, st);
    else state_partial<float, 128>(m, c, k_new, v_new, max_new, n_new, ws, base, st);
  } else {
    if (m.d == 64) state_partial<bf16_t, 64>(m, c, k_new, v_new, max_new, n_new, ws, base, st);
    else state_partial<bf16_t, 128>(m, c, k_new, v_new, max_new, n_new, ws, base, st);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(append_state_reduce_kernel, dim3(m.d / kReduceRows, m.bh), dim3(256), 0,
                     st, m, ws.n_chunks, (const float*)(base + ws.part_s),
                     (const float*)(base + ws.part_z), c.lin_state, c.lin_norm, nullptr, 0,
                     nullptr);
  return hipGetLastError();
}

bool append_fusable(const Dims& m) { return m.elem == 2 && m.d == 128 && !windowed(m); }

hipError_t launch_append_fused(const Dims& m, const spla_cache& c, const void* k_new,
                               const void* v_new, int max_new, const int32_t* n_new,
                               const AppendWs& ws, char* base, hipStream_t st) {
  if (!append_fusable(m)) return hipErrorInvalidValue;
  // block-aligned chunks: the first starts up to B - 1 positions before the
  // append point, so n_chunks chunks of ct tokens cover B - 1 + max_new
  const int ct = (int)align_up(ceil_div((int64_t)max_new + m.B - 1, ws.n_chunks),
                               m.B > kSubTokens ? m.B : kSubTokens);
  hipLaunchKernelGGL(append_fused_kernel<128>, dim3(ws.n_chunks, m.bh), dim3(256), 0, st, m,
                     (bf16_t*)c.k_cache, (bf16_t*)c.v_cache, c.blk_stats, c.seq_lens, c.err_flags,
                     (const bf16_t*)k_new, (const bf16_t*)v_new, max_new, n_new,
                     m.pages > 0 ? c.block_table : nullptr, ws.n_chunks, ct,
                     (float*)(base + ws.part_s), (float*)(base + ws.part_z));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(append_state_reduce_kernel, dim3(m.d / kReduceRows, m.bh), dim3(256), 0,
                     st, m, ws.n_chunks, (const float*)(base + ws.part_s),
                     (const float*)(base + ws.part_z), c.lin_state, c.lin_norm, c.seq_lens,
                     max_new, n_new);
  return hipGetLastError();
}

// Units a single token touches: one block, or up to ul / us windows.
static int64_t units_of_one(const Dims& m) { return windowed(m) ? m.ul / m.us : 1; }

template <typename T, int D>
static void append_one_td(const Dims& m, const spla_cache& c, const void* k_new,
                          const void* v_new, hipStream_t st, bool rank1, int32_t* fin_ctr,
                          int32_t* appended) {
  if (!rank1) {  // statistics and rows only
    hipLaunchKernelGGL(append_unit_kernel<T>, dim3((unsigned)units_of_one(m), (unsigned)m.bh),
                       dim3(D), 0, st, m, (T*)c.k_cache, (T*)c.v_cache, c.blk_stats, c.seq_lens,
                       c.err_flags, (const T*)k_new, (const T*)v_new,
                       m.pages > 0 ? c.block_table : nullptr, fin_ctr, appended);
    return;
  }
  hipLaunchKernelGGL((append_one_kernel<T, D>), dim3((unsigned)(D / 16 + units_of_one(m)),
                     (unsigned)m.bh), dim3(256), 0, st, m, (T*)c.k_cache, (T*)c.v_cache,
                     c.blk_stats, c.seq_lens, c.err_flags, (const T*)k_new, (const T*)v_new,
                     m.pages > 0 ? c.block_table : nullptr, c.lin_state, c.lin_norm, fin_ctr,
                     appended);
}

hipError_t launch_append_one(const Dims& m, const spla_cache& c, const void* k_new,
                             const void* v_new, hipStream_t st, bool rank1, int32_t* fin_ctr,
                             int32_t* appended) {
  if (m.elem == 4) {
    if (m.d == 64) append_one_td<float, 64>(m, c, k_new, v_new, st, rank1, fin_ctr, appended);
    else append_one_td<float, 128>(m, c, k_new, v_new, st, rank1, fin_ctr, appended);
  } else {
    if (m.d == 64) append_one_td<bf16_t, 64>(m, c, k_new, v_new, st, rank1, fin_ctr, appended);
    else append_one_td<bf16_t, 128>(m, c, k_new, v_new, st, rank1, fin_ctr, appended);
  }
  return hipGetLastError();
}

hipError_t launch_append_finish(const Dims& m, const spla_cache& c, int max_new,
                                const int32_t* n_new, hipStream_t st, int32_t* appended) {
  hipLaunchKernelGGL(append_finish_kernel, dim3((unsigned)ceil_div(m.batch, 256)), dim3(256), 0,
                     st, m, c.seq_lens, max_new, n_new, appended);
  return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t st) {
  const int64_t n = (int64_t)(bytes / 4);
  if (n == 0) return hipSuccess;
  int64_t blocks = ceil_div(n, 256);
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, st, (uint32_t*)p, n);
  return hipGetLastError();
}

}  // namespace spla
