// Device kernels of the batched inference path, written for gfx950 (CDNA4,
// wave64, MFMA, 160 KB LDS per CU).
//
// A launch group is a set of dispatched batches of one queue. Its rows live in
// one row space: batch b owns rows [row_base_b, row_base_b + P_b), the first
// s_b of them real, the rest padding (the batch axis padded to an allowed
// size). The kernels, in the order a group runs them:
//
//   route     per-batch exclusive prefix scans: which request row (or padding)
//             every row is, where its input and output live (the paper's
//             concatenation of input tensors, section 2.2.1, as an index map)
//   assemble  gather request rows into the padded batch tensor (optional
//             fp32 -> bf16 cast), or
//   embbag    sum-pool each row's embedding bags (ranking models)
//   gemm      dense layers with fused bias + activation (bf16 or fp32 MFMA);
//             the last layer of a chain without a head writes its real rows
//             straight into the requests' outputs through the row map (the
//             split fused in)
//   gemm_head the last hidden layer of 256 outputs and a narrow head in one
//             kernel, or
//   head /    narrow last layer or masked mean-pool + softmax head, writing
//   seqpool   straight to each request's output rows
//   split     copy real rows to their requests' outputs (padding dropped;
//             the unfused form, kept for the C ABI)
//
// Every row is computed the same way whatever batch it sits in (one tile
// shape and k order per layer, no row-count-dependent split of the sum), so a
// request's result does not depend on how its batch was composed.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <algorithm>
#include <atomic>
#include <mutex>

#include "../../include/rb.h"

namespace {

typedef uint16_t bf16_t;
typedef __attribute__((__vector_size__(8 * sizeof(short)))) short bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16_t;
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef int i32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ bf16_t f2bf(float f) {
  // round to nearest even on the 16 dropped bits; NaN stays a (quiet) NaN
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

__device__ __forceinline__ float bf2f(uint32_t h) { return __uint_as_float(h << 16); }

__device__ __forceinline__ uint32_t pack2(float a, float b) {
  return (uint32_t)f2bf(a) | ((uint32_t)f2bf(b) << 16);
}

template <int ACT>
__device__ __forceinline__ float act_fn(float z) {
  if (ACT == RB_ACT_RELU) return z > 0.f ? z : 0.f;
  if (ACT == RB_ACT_SIGMOID) return 1.f / (1.f + expf(-z));
  return z;
}

// Workgroups are handed to the 8 XCDs round-robin (block i runs on XCD i % 8)
// and each XCD has its own L2. Remap so that XCD x gets a contiguous range of
// tiles: with tiles ordered row-block-major, the tiles sharing an A row-block
// then run on the same XCD and re-read it from that XCD's L2.
__device__ __forceinline__ int xcd_tile(int bid, int nb) {
  const int nb8 = nb & ~7;
  return bid < nb8 ? (bid & 7) * (nb8 >> 3) + (bid >> 3) : bid;
}

__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// ---------------------------------------------------------------- route

constexpr int ROUTE_MAX_ROWS = 4096;  // rows (sequence slots) per batch

// Block-wide exclusive scan of one value per thread (256 threads); returns
// the exclusive prefix and writes the block total to *total.
__device__ __forceinline__ int64_t block_exclusive_scan(int64_t v, int64_t* s_w, int64_t* total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  int64_t incl = v;
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t u = __shfl_up(incl, o);
    if (lane >= o) incl += u;
  }
  if (lane == 63) s_w[wid] = incl;
  __syncthreads();
  int64_t off = 0;
  for (int w = 0; w < wid; ++w) off += s_w[w];
  *total = s_w[0] + s_w[1] + s_w[2] + s_w[3];
  __syncthreads();
  return off + incl - v;
}

// One workgroup per batch, all steps parallel over requests or rows:
//  1. exclusive scan of the requests' row counts -> each request's first row
//     (the concatenation offsets), and a row -> request map in LDS;
//  2. per real row, its id count (ranking: sum of its bag lengths) or token
//     count (seqpool: its sequence length), loaded in parallel;
//  3. exclusive scan of those counts over the batch's rows; a row's first id
//     (token) is its request's base plus the scan difference to the request's
//     first row; each request is checked against its payload extent;
//  4. the row map entries, then padding rows. A sequence's entry also names
//     the row of its first token when the group's real tokens are packed
//     (its request's first packed row, set by the host, plus the scan).
__global__ __launch_bounds__(256) void k_route(int kind, const rb_k_batch* __restrict__ batches,
                                               const rb_k_req* __restrict__ reqs, int n_reqs,
                                               const int32_t* __restrict__ lens, int64_t lens_len, int d_in,
                                               int d_out, int n_tables, rb_k_row* __restrict__ rows,
                                               int n_rows_total, int64_t out_len, int* __restrict__ err) {
  const rb_k_batch b = batches[blockIdx.x];
  const int tid = threadIdx.x;
  __shared__ int s_first[ROUTE_MAX_ROWS + 1];   // first row of request i (batch-relative)
  __shared__ int s_req[ROUTE_MAX_ROWS];         // request of row p
  __shared__ int64_t s_ex[ROUTE_MAX_ROWS + 1];  // exclusive scan of per-row id/token counts
  __shared__ unsigned char s_bad[ROUTE_MAX_ROWS];
  __shared__ int64_t s_w[4];
  // the batch's rows and requests must lie inside the row map and the
  // request table (its rows are then left as they are)
  if (b.padded > ROUTE_MAX_ROWS || b.n_req > b.padded || b.real > b.padded || b.padded < 0 || b.n_req < 0 ||
      b.row_base < 0 || (int64_t)b.row_base + b.padded > n_rows_total || b.req_begin < 0 ||
      (int64_t)b.req_begin + b.n_req > n_reqs) {
    if (tid == 0) *err = 1;
    return;
  }
  // 1. request offsets
  __shared__ int s_desc_bad;
  if (tid == 0) s_desc_bad = 0;
  __syncthreads();
  int64_t carry = 0;
  for (int base = 0; base < b.n_req; base += 256) {
    const int i = base + tid;
    const int n = i < b.n_req ? reqs[b.req_begin + i].n_rows : 0;
    if (i < b.n_req && n < 1) s_desc_bad = 1;  // every request has >= 1 row
    int64_t tot;
    const int64_t ex = block_exclusive_scan(n, s_w, &tot);
    if (i < b.n_req) {
      s_first[i] = (int)(carry + ex);
      s_bad[i] = 0;
    }
    carry += tot;
  }
  if (tid == 0) s_first[b.n_req] = (int)carry;
  __syncthreads();
  const int s = (int)carry;
  if (s > b.padded || s_desc_bad) {
    if (tid == 0) *err = 1;
    return;
  }
  for (int i = tid; i < b.n_req; i += 256)
    for (int p = s_first[i]; p < s_first[i + 1]; ++p) s_req[p] = i;
  __syncthreads();
  // 2 + 3. per-row counts and their scan
  carry = 0;
  for (int base = 0; base < s; base += 256) {
    const int p = base + tid;
    int64_t c = 0;
    if (p < s) {
      const int i = s_req[p];
      const rb_k_req& rq = reqs[b.req_begin + i];
      const int e = p - s_first[i];
      // a request whose output rows would lie outside the output, or whose bag
      // or sequence lengths outside the lens arena, is rejected
      const int64_t nl = kind == RB_MODEL_RANKING ? (int64_t)rq.n_rows * n_tables
                                                  : (kind == RB_MODEL_SEQPOOL ? rq.n_rows : 0);
      const bool in_arena = e < rq.n_rows && rq.out_off >= 0 && rq.out_off + (int64_t)rq.n_rows * d_out <= out_len &&
                            (nl == 0 || (rq.lens_off >= 0 && rq.lens_off + nl <= lens_len));
      if (!in_arena) {
        s_bad[i] = 1;
      } else if (kind == RB_MODEL_MLP) {
      } else if (kind == RB_MODEL_RANKING) {
        const int32_t* l = lens + rq.lens_off + (int64_t)e * n_tables;
        // the flag is kept in a register so that the unrolled loads are all
        // issued before the first one is used
        bool neg = false;
#pragma unroll 8
        for (int f = 0; f < n_tables; ++f) {
          const int v = l[f];
          neg |= v < 0;
          c += v;
        }
        if (neg) s_bad[i] = 1;
      } else {
        const int v = lens[rq.lens_off + e];
        if (v < 1 || v > b.seq_T) s_bad[i] = 1;
        c = v;
      }
    }
    int64_t tot;
    const int64_t ex = block_exclusive_scan(c, s_w, &tot);
    if (p < s) s_ex[p] = carry + ex;
    carry += tot;
  }
  if (tid == 0) s_ex[s] = carry;
  __syncthreads();
  for (int i = tid; i < b.n_req; i += 256) {
    const rb_k_req& rq = reqs[b.req_begin + i];
    const int n = s_first[i + 1] - s_first[i];
    const int64_t cnt = s_ex[s_first[i + 1]] - s_ex[s_first[i]];
    bool ok = !s_bad[i] && n == rq.n_rows;
    if (kind == RB_MODEL_SEQPOOL) ok = ok && cnt * d_in == rq.dense_end - rq.dense_off;
    else ok = ok && (int64_t)n * d_in == rq.dense_end - rq.dense_off;
    if (kind == RB_MODEL_RANKING) ok = ok && cnt == rq.ids_end - rq.ids_off;
    if (!ok) *err = 1;
    s_bad[i] = ok ? 0 : 1;
  }
  __syncthreads();
  // 4. row entries
  for (int p = tid; p < b.padded; p += 256) {
    rb_k_row rw;
    if (p < s) {
      const int i = s_req[p];
      const rb_k_req& rq = reqs[b.req_begin + i];
      const int e = p - s_first[i];
      const bool ok = !s_bad[i];
      const int64_t within = s_ex[p] - s_ex[s_first[i]];
      if (kind == RB_MODEL_SEQPOOL) {
        rw.src = ok ? rq.dense_off + within * d_in : -1;
        rw.aux = ok ? s_ex[p + 1] - s_ex[p] : 0;
        rw.lens = ok ? rq.tok_off + within : -1;  // first row among the group's packed tokens
      } else {
        rw.src = ok ? rq.dense_off + (int64_t)e * d_in : -1;
        rw.aux = rq.ids_off + within;
        rw.lens = (kind == RB_MODEL_RANKING && ok) ? rq.lens_off + (int64_t)e * n_tables : -1;
      }
      rw.out = ok ? rq.out_off + (int64_t)e * d_out : -1;  // a rejected request's rows are not returned
    } else {
      rw.src = -1;
      rw.aux = 0;
      rw.lens = -1;
      rw.out = -1;
    }
    rows[b.row_base + p] = rw;
  }
}

// ---------------------------------------------------------------- assemble

// One thread per 8 output elements of a row: coalesced 16-byte stores of the
// padded batch tensor. Padding rows (and padding tokens) get `pad` in their
// d_in input columns; columns past d_in are always zero so that they add
// nothing in the next contraction.
// Real tokens only (sequence slots): workgroup (e, j) copies tokens
// [16 j, 16 j + 16) of slot e that lie below its length L (8 columns per thread
// and chunk, two chunks in flight, columns past d_in zeroed); blocks past L,
// rows t >= L and padding slots are not written (8..64-token blocks and 1..4
// chunks in flight measured no faster). Token t goes to row e T + t of X, or,
// with PACKED, to row rows[e].lens + t of the group's packed tokens (x_rows
// rows). lg_c = log2(ldx / 8) when that is a power of two, else -1.
constexpr int SEQ_TOK = 16, SEQ_U = 2;
template <bool PACKED>
__global__ __launch_bounds__(256) void k_assemble_seq(const rb_k_row* __restrict__ rows, int T,
                                                      const float* __restrict__ dense, int64_t dense_len, int d_in,
                                                      float* __restrict__ X, int ldx, int64_t x_rows,
                                                      int* __restrict__ err, int lg_c) {
  const rb_k_row rw = rows[blockIdx.x];
  const int t0 = blockIdx.y * SEQ_TOK;
  if (rw.src < 0 || t0 >= rw.aux) return;
  const int64_t L = rw.aux;
  if (L > T || rw.src + L * d_in > dense_len || (PACKED && (rw.lens < 0 || rw.lens + L > x_rows))) {
    if (threadIdx.x == 0) *err = 1;
    return;
  }
  const int cpr = ldx >> 3;
  const int n_tok = (int)min((int64_t)SEQ_TOK, L - t0);
  const int total = n_tok * cpr;
  const float* src = dense + rw.src + (int64_t)t0 * d_in;
  float* xb = X + ((PACKED ? rw.lens : (int64_t)blockIdx.x * T) + t0) * ldx;
  const bool vec = (d_in & 3) == 0 && (rw.src & 3) == 0;
  // SEQ_U chunks per thread and step: all loads issued before the stores
  for (int base = threadIdx.x; base < total; base += 256 * SEQ_U) {
    float v[SEQ_U][8];
#pragma unroll
    for (int u = 0; u < SEQ_U; ++u) {
      const int i = base + 256 * u;
      if (i >= total) break;
      const int t = lg_c >= 0 ? i >> lg_c : i / cpr;
      const int c0 = (i - t * cpr) * 8;
      const float* sr = src + (int64_t)t * d_in;
      if (vec) {
#pragma unroll
        for (int h = 0; h < 8; h += 4) {
          if (c0 + h < d_in) {
            const float4 a = *(const float4*)(sr + c0 + h);
            v[u][h] = a.x; v[u][h + 1] = a.y; v[u][h + 2] = a.z; v[u][h + 3] = a.w;
          } else {
            v[u][h] = v[u][h + 1] = v[u][h + 2] = v[u][h + 3] = 0.f;
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j) v[u][j] = (c0 + j < d_in) ? sr[c0 + j] : 0.f;
      }
    }
#pragma unroll
    for (int u = 0; u < SEQ_U; ++u) {
      const int i = base + 256 * u;
      if (i >= total) break;
      const int t = lg_c >= 0 ? i >> lg_c : i / cpr;
      const int c0 = (i - t * cpr) * 8;
      float* y = xb + (int64_t)t * ldx + c0;
      *(float4*)y = make_float4(v[u][0], v[u][1], v[u][2], v[u][3]);
      *(float4*)(y + 4) = make_float4(v[u][4], v[u][5], v[u][6], v[u][7]);
    }
  }
}

// One thread per 8 consecutive columns of one row (one 16-byte bf16 store or
// two fp32 ones; 4 or 16 columns measured slower). POW2: ldx / 8 and seq_T
// (when non-zero) are powers of two and the thread count fits 31 bits, so the
// row, chunk and slot indices come from shifts (lg_c = log2(ldx / 8), lg_t =
// log2(seq_T)); otherwise 64-bit division.
template <bool BF16, bool POW2>
__global__ __launch_bounds__(256) void k_assemble(const rb_k_row* __restrict__ rows, int n_rows_total,
                                                  int seq_T, const float* __restrict__ dense,
                                                  int64_t dense_len, int d_in, void* __restrict__ X,
                                                  int ldx, float pad, int* __restrict__ err, int lg_c, int lg_t) {
  constexpr int E = 8;
  const int chunks = ldx / E;
  int64_t r;
  int c0;
  if (POW2) {
    const uint32_t gid = blockIdx.x * 256u + threadIdx.x;
    r = (int64_t)(gid >> lg_c);
    c0 = (int)(gid & (uint32_t)(chunks - 1)) * E;
  } else {
    const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
    r = gid / chunks;
    c0 = (int)(gid - r * chunks) * E;
  }
  if (r >= n_rows_total) return;
  int64_t src;
  if (seq_T > 0) {
    const int64_t slot = POW2 ? (int64_t)((uint32_t)r >> lg_t) : r / seq_T;
    const int t = (int)(r - slot * seq_T);
    const rb_k_row rw = rows[slot];
    src = (rw.src >= 0 && t < rw.aux) ? rw.src + (int64_t)t * d_in : -1;
  } else {
    src = rows[r].src;
  }
  float v[E];
  if (src < 0) {
#pragma unroll
    for (int j = 0; j < E; ++j) v[j] = (c0 + j < d_in) ? pad : 0.f;
  } else if (src + d_in > dense_len) {
    *err = 1;
#pragma unroll
    for (int j = 0; j < E; ++j) v[j] = 0.f;
  } else if ((d_in & 3) == 0 && (src & 3) == 0) {
#pragma unroll
    for (int h = 0; h < E; h += 4) {
      if (c0 + h < d_in) {  // d_in % 4 == 0: all 4 columns are inputs
        const float4 a = *(const float4*)(dense + src + c0 + h);
        v[h + 0] = a.x; v[h + 1] = a.y; v[h + 2] = a.z; v[h + 3] = a.w;
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) v[h + j] = 0.f;
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < E; ++j) v[j] = (c0 + j < d_in) ? dense[src + c0 + j] : 0.f;
  }
  if (BF16) {
    bf16_t* y = (bf16_t*)X + r * ldx + c0;
    *(uint4*)y = make_uint4(pack2(v[0], v[1]), pack2(v[2], v[3]), pack2(v[4], v[5]), pack2(v[6], v[7]));
  } else {
    float* y = (float*)X + r * ldx + c0;
#pragma unroll
    for (int h = 0; h < E; h += 4) *(float4*)(y + h) = make_float4(v[h], v[h + 1], v[h + 2], v[h + 3]);
  }
}

// ---------------------------------------------------------------- embedding bags

constexpr int EMB_DIM = 64;       // one table row = 128 bytes of bf16
constexpr int MAX_TABLES = 64;
constexpr int EMB_SLICES = MAX_TABLES;  // table slices: one table each (up to MAX_TABLES)
constexpr int EMB_CHUNK = 8;      // ids loaded (one per lane of a group) and gathers issued per round
static_assert(EMB_CHUNK <= 8, "each of a group's 8 lanes loads one id of a chunk");
// (4 ids per round measured 4% slower; 16 or 24, two or three per lane, 1.5x
// and 1.7x slower; fewer workgroups per CU, capped through LDS, 1.25x to 2.8x
// slower: the gather wants every load in flight the registers can hold)

// One 8-lane group per (row, bag); lane l8 owns dims [8 l8, 8 l8 + 8) of the
// 64-dim table rows. The grid is slice-major: workgroups [x nrb, (x + 1) nrb)
// serve table slice x (tables x, x + n_slices, ...; with one table per slice,
// table x) for rpw consecutive rows each, so at any time the whole chip
// gathers from one or two tables and every XCD's L2 and the Infinity Cache
// hold their hot rows (all tables at once per row measured 1.5x slower, 4 or
// 8 slices 1.2x slower).
// A group finds its bag in the row's flat id list (bag after bag) with an
// 8-lane sum of the preceding bag lengths; the row-map entry takes one round
// trip and all the lengths one more (loaded one after another, as a loop that
// adds each length as it arrives compiles, they took up to five: the kernel
// was 4-5% slower on one box). The workgroup's 32 bags are then
// ranked by length through LDS and the group of rank p walks the bag of rank
// p, so the 8 bags of a wave have similar lengths and its gather instructions
// keep most lanes busy (uniform 1..20-id bags: 50 gather instructions per
// workgroup instead of 73; 2-3% faster). A bag is walked EMB_CHUNK ids at a
// time: lane i loads id c + i, the ids are broadcast within the group and all
// EMB_CHUNK gathers are issued before any is added. Sums are fp32 in id order
// (a fixed order that depends on the bag only), stored as bf16. The workgroups
// of slice 0 also write the rows' dense features and zero tails.
// Reads stay inside the ids arena and the tables: an id position past the
// arena or an id outside its table sets *err = 1 and contributes nothing.
__global__ __launch_bounds__(256) void k_embbag(const rb_k_row* __restrict__ rows, int n_rows,
                                                const int32_t* __restrict__ lens,
                                                const int32_t* __restrict__ ids, int64_t ids_len,
                                                const bf16_t* const* __restrict__ tables, int n_tables,
                                                int64_t table_rows, const float* __restrict__ dense,
                                                int n_dense, bf16_t* __restrict__ X, int ldx, int n_slices,
                                                int gpr, int rpw, float pad, int* __restrict__ err) {
  const int nrb = gridDim.x / n_slices;  // row blocks per slice
  const int x = blockIdx.x / nrb;
  const int r0 = (blockIdx.x - x * nrb) * rpw;
  const int tid = threadIdx.x, g = tid >> 3, l8 = tid & 7;
  const int gbase = (tid & 63) & ~7;  // this group's first lane in the wave
  const int demb = n_tables * EMB_DIM;
  // 1. group g's own bag: its length (-1: no bag, -2: a padding row) and its
  //    first id's position in the ids arena
  __shared__ int s_key[32];
  __shared__ int s_bag[32], s_len[32];
  __shared__ int64_t s_id0[32];
  int L = -1;
  int64_t id0 = 0;
  {
    const int row = r0 + g / gpr, t = x + n_slices * (g % gpr);
    if (g < rpw * gpr && row < n_rows && t < n_tables) {
      // the 32-byte entry as two 16-byte loads issued together (the empty asm
      // uses the second half here, so that its load is not moved after the
      // test of the first half and waited for separately)
      const u32x4_t* re = (const u32x4_t*)(rows + row);
      const u32x4_t e0 = re[0], e1 = re[1];
      asm volatile("" ::"v"(e1.x), "v"(e1.y));
      rb_k_row rw;
      rw.src = (int64_t)((uint64_t)e0.x | ((uint64_t)e0.y << 32));
      rw.aux = (int64_t)((uint64_t)e0.z | ((uint64_t)e0.w << 32));
      rw.lens = (int64_t)((uint64_t)e1.x | ((uint64_t)e1.y << 32));
      if (rw.src < 0) {
        L = -2;
      } else {
        // lane l8 loads the lengths of tables l8, l8 + 8, ... below t and
        // the bag's own length, all issued before any is used (a loop that
        // adds each length as it arrives waits for every load in turn)
        int v[MAX_TABLES / 8];
#pragma unroll
        for (int u = 0; u < MAX_TABLES / 8; ++u) {
          const int f = l8 + 8 * u;
          v[u] = f < t ? lens[rw.lens + f] : 0;
        }
        L = lens[rw.lens + t];
        int pre = 0;
#pragma unroll
        for (int u = 0; u < MAX_TABLES / 8; ++u) pre += v[u];
        pre += __shfl_xor(pre, 1);
        pre += __shfl_xor(pre, 2);
        pre += __shfl_xor(pre, 4);
        id0 = rw.aux + pre;
      }
    }
  }
  // 2. the workgroup's 32 bags ranked longest first (ties by group), and
  //    group p takes the bag of rank p: the 8 bags of a wave then have
  //    similar lengths, so its gather instructions keep most lanes busy
  if (l8 == 0) s_key[g] = L;
  __syncthreads();
  {
    int rank = 0;
    for (int h = l8; h < 32; h += 8) {
      const int k = s_key[h];
      rank += (k > L || (k == L && h < g)) ? 1 : 0;
    }
    rank += __shfl_xor(rank, 1);
    rank += __shfl_xor(rank, 2);
    rank += __shfl_xor(rank, 4);
    if (l8 == 0) {
      s_bag[rank] = g;
      s_len[rank] = L;
      s_id0[rank] = id0;
    }
  }
  __syncthreads();
  const int b = s_bag[g];
  L = s_len[g];
  id0 = s_id0[g];
  // 3. the bag's walk
  if (L != -1) {
    const int row = r0 + b / gpr, t = x + n_slices * (b % gpr);
    u32x4_t o;
    if (L == -2) {
      const uint32_t p = f2bf(pad);
      o = (u32x4_t){p | (p << 16), p | (p << 16), p | (p << 16), p | (p << 16)};
    } else {
      const bf16_t* tab = tables[t];
      float acc[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) acc[k] = 0.f;
      // lane i's id of chunk c (-1: past the bag or outside the ids arena)
      auto chunk_id = [&](int c) {
        const int64_t pos = id0 + c + l8;
        return (c + l8 < L && pos >= 0 && pos < ids_len) ? ids[pos] : -1;
      };
      int nxt = chunk_id(0);
      for (int c = 0; c < L; c += EMB_CHUNK) {
        const int my = nxt;
        nxt = chunk_id(c + EMB_CHUNK);  // the next chunk's ids load during this chunk's gathers
        u32x4_t q[EMB_CHUNK];
#pragma unroll
        for (int u = 0; u < EMB_CHUNK; ++u) {
          const int id = __shfl(my, gbase + u);
          q[u] = (u32x4_t){0u, 0u, 0u, 0u};
          if (c + u < L) {
            if ((uint64_t)(int64_t)id < (uint64_t)table_rows)
              q[u] = *(const u32x4_t*)(tab + (int64_t)id * EMB_DIM + l8 * 8);
            else
              *err = 1;
          }
        }
#pragma unroll
        for (int u = 0; u < EMB_CHUNK; ++u) {
          acc[0] += bf2f(q[u].x & 0xffffu); acc[1] += bf2f(q[u].x >> 16);
          acc[2] += bf2f(q[u].y & 0xffffu); acc[3] += bf2f(q[u].y >> 16);
          acc[4] += bf2f(q[u].z & 0xffffu); acc[5] += bf2f(q[u].z >> 16);
          acc[6] += bf2f(q[u].w & 0xffffu); acc[7] += bf2f(q[u].w >> 16);
        }
      }
      o.x = pack2(acc[0], acc[1]);
      o.y = pack2(acc[2], acc[3]);
      o.z = pack2(acc[4], acc[5]);
      o.w = pack2(acc[6], acc[7]);
    }
    *(u32x4_t*)(X + (int64_t)row * ldx + t * EMB_DIM + l8 * 8) = o;
  }
  if (x == 0) {
    // the dense features and zero tail (columns demb .. ldx, a multiple of 8
    // wide): one 8-column chunk, a 16-byte store, per thread and pass, so that
    // the loads of all the block's rows are in flight at once
    const int cpr = (ldx - demb) >> 3;
    for (int e = tid; e < rpw * cpr; e += 256) {
      const int i = e / cpr, c = e - i * cpr;
      if (r0 + i >= n_rows) break;
      const rb_k_row rw = rows[r0 + i];
      uint32_t h[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int d = 8 * c + k;
        h[k] = d < n_dense ? (uint32_t)f2bf(rw.src < 0 ? pad : dense[rw.src + d]) : 0u;
      }
      const u32x4_t o = {h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
      *(u32x4_t*)(X + (int64_t)(r0 + i) * ldx + demb + 8 * c) = o;
    }
  }
}

// Embedding bags with the ids of a batch block deduplicated per table
// (compressing away features common to a batch of examples, paper section
// 2.2): workgroup (table t, block of DD_ROWS rows) stages the block's bag ids
// for table t in LDS, finds the distinct ones with an open-addressing hash in
// LDS, gathers each distinct table row once into LDS (up to DD_UCAP rows,
// 128 bytes each, 16-byte loads by 8-lane groups), then sums every bag from
// LDS in id order. The sums are the same fp32 additions in the same order as
// k_embbag's, so the outputs are bit-identical; only the table rows gathered
// per block change (measured on the ranking workload: 672 ids per 64-row block
// and table, 345 distinct). Ids past DD_NMAX positions in the block, or
// distinct rows past DD_UCAP, are gathered from the table directly. The same
// bounds as k_embbag: an id position outside the ids arena or an id outside its
// table sets *err = 1 and contributes +0.
constexpr int DD_ROWS = 64;     // rows per workgroup
constexpr int DD_NT = 512;      // threads per workgroup: 8 per row, 64 8-lane groups
constexpr int DD_NMAX = 1280;   // id positions staged per workgroup (64 rows x 20 ids)
constexpr int DD_HS = 2048;     // hash slots (> DD_NMAX: an insert always finds a free slot)
constexpr int DD_UCAP = 448;    // distinct table rows staged per workgroup (56 KB)

__global__ __launch_bounds__(DD_NT) void k_embbag_dedup(const rb_k_row* __restrict__ rows, int n_rows,
                                                        const int32_t* __restrict__ lens,
                                                        const int32_t* __restrict__ ids, int64_t ids_len,
                                                        const bf16_t* const* __restrict__ tables, int n_tables,
                                                        int64_t table_rows, const float* __restrict__ dense,
                                                        int n_dense, bf16_t* __restrict__ X, int ldx, float pad,
                                                        int* __restrict__ err) {
  __shared__ u32x4_t s_u[DD_UCAP][8];   // distinct table rows (8 x 16 bytes each)
  __shared__ int32_t s_key[DD_HS];      // hash slot -> table row id (-1: empty)
  __shared__ int16_t s_slot[DD_HS];     // hash slot -> distinct-row index
  __shared__ int32_t s_ids[DD_NMAX];    // the block's ids, bag after bag (-1: invalid)
  __shared__ int16_t s_k[DD_NMAX];      // id position -> hash slot, then -> distinct-row index (-1: invalid)
  __shared__ int32_t s_uid[DD_UCAP];    // distinct-row index -> table row id
  __shared__ int32_t s_len[DD_ROWS], s_start[DD_ROWS + 1];
  __shared__ int64_t s_id0[DD_ROWS];    // a row's first id of table t in the ids arena
  __shared__ int s_wsum[DD_NT / 64];
  const int nrb = gridDim.x / n_tables;
  const int t = blockIdx.x / nrb;
  const int r0 = (blockIdx.x - t * nrb) * DD_ROWS;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int g = tid >> 3, l8 = tid & 7;  // 8-lane group g serves row g
  const bf16_t* tab = tables[t];
  for (int h = tid; h < DD_HS; h += DD_NT) s_key[h] = -1;
  // 1. row g's bag of table t: its 8 lanes load the row's bag lengths
  //    (lane l8 those of tables l8, l8 + 8, ... below t, all at once) and sum
  //    them; then an exclusive scan over the block's rows
  {
    int pre = 0, L = 0;
    int64_t aux = 0;
    bool real = false;
    if (r0 + g < n_rows) {
      const rb_k_row rw = rows[r0 + g];
      real = rw.src >= 0;
      if (real) {
        int v[MAX_TABLES / 8];
#pragma unroll
        for (int u = 0; u < MAX_TABLES / 8; ++u) {
          const int f = l8 + 8 * u;
          v[u] = f < t ? lens[rw.lens + f] : 0;
        }
#pragma unroll
        for (int u = 0; u < MAX_TABLES / 8; ++u) pre += v[u];
        L = lens[rw.lens + t];
        aux = rw.aux;
      }
    }
    pre += __shfl_xor(pre, 1);
    pre += __shfl_xor(pre, 2);
    pre += __shfl_xor(pre, 4);
    if (l8 == 0) {
      s_len[g] = real ? max(L, 0) : 0;
      s_id0[g] = aux + pre;
    }
  }
  __syncthreads();
  if (wid == 0) {  // exclusive scan of the 64 bag lengths
    const int v = s_len[lane];
    int incl = v;
    for (int o = 1; o < 64; o <<= 1) {
      const int u = __shfl_up(incl, o);
      if (lane >= o) incl += u;
    }
    s_start[lane] = incl - v;
    if (lane == 63) s_start[DD_ROWS] = incl;
  }
  __syncthreads();
  const int n_pos = min(s_start[DD_ROWS], DD_NMAX);
  // 2. stage the ids: row g's 8 lanes take its bag's positions l8, l8 + 8, ...
  {
    const int L = s_len[g], st = s_start[g];
    const int64_t id0 = s_id0[g];
    for (int j0 = 0; j0 < L && st + j0 < DD_NMAX; j0 += 32) {
      int v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = j0 + l8 + 8 * u;
        const int64_t pos = id0 + j;
        v[u] = (j < L && pos >= 0 && pos < ids_len) ? ids[pos] : -1;
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int j = j0 + l8 + 8 * u;
        if (j < L && st + j < DD_NMAX) {
          int id = v[u];
          if ((uint64_t)(int64_t)id >= (uint64_t)table_rows) {
            *err = 1;
            id = -1;
          }
          s_ids[st + j] = id;
        }
      }
    }
  }
  __syncthreads();
  // 3. distinct ids: insert every staged id into the hash (linear probing)
  for (int i = tid; i < n_pos; i += DD_NT) {
    const int id = s_ids[i];
    int h = -1;
    if (id >= 0) {
      h = (int)(((uint32_t)id * 2654435761u) >> 21);  // 11 bits: DD_HS slots
      for (;;) {
        const int old = atomicCAS(&s_key[h], -1, id);
        if (old == -1 || old == id) break;
        h = (h + 1) & (DD_HS - 1);
      }
    }
    s_k[i] = (int16_t)h;
  }
  __syncthreads();
  // 4. number the occupied slots (block scan, 4 slots per thread)
  {
    constexpr int SPT = DD_HS / DD_NT;
    int occ[SPT], c = 0;
#pragma unroll
    for (int k = 0; k < SPT; ++k) {
      occ[k] = s_key[tid * SPT + k] >= 0;
      c += occ[k];
    }
    int incl = c;
    for (int o = 1; o < 64; o <<= 1) {
      const int u = __shfl_up(incl, o);
      if (lane >= o) incl += u;
    }
    if (lane == 63) s_wsum[wid] = incl;
    __syncthreads();
    int base = incl - c;
    for (int w = 0; w < wid; ++w) base += s_wsum[w];
#pragma unroll
    for (int k = 0; k < SPT; ++k) {
      if (occ[k]) {
        s_slot[tid * SPT + k] = (int16_t)base;
        if (base < DD_UCAP) s_uid[base] = s_key[tid * SPT + k];
        ++base;
      }
    }
  }
  __syncthreads();
  int n_all = 0;
#pragma unroll
  for (int w = 0; w < DD_NT / 64; ++w) n_all += s_wsum[w];
  const int n_u = min(n_all, DD_UCAP);
  // 5. every distinct row once (8-lane group g: rows g, g + 64, ...), and each
  //    staged position's distinct-row index (hash slot replaced by it)
  {
    constexpr int UNR = 4;
    for (int k0 = g; k0 < n_u; k0 += (DD_NT / 8) * UNR) {
      u32x4_t v[UNR];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int k = k0 + (DD_NT / 8) * u;
        if (k < n_u) v[u] = *(const u32x4_t*)(tab + (int64_t)s_uid[k] * EMB_DIM + l8 * 8);
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int k = k0 + (DD_NT / 8) * u;
        if (k < n_u) s_u[k][l8] = v[u];
      }
    }
    for (int i = tid; i < n_pos; i += DD_NT) {
      const int h = s_k[i];
      // rows past the staged ones keep -2 - hash slot: gathered directly
      s_k[i] = (int16_t)(h < 0 ? -1 : (s_slot[h] < DD_UCAP ? s_slot[h] : -2 - h));
    }
  }
  __syncthreads();
  // 6. row g's bag from the staged rows, in id order (fp32), stored as bf16;
  //    8 ids per round, their reads issued before any is added
  if (r0 + g < n_rows) {
    const rb_k_row rw = rows[r0 + g];
    u32x4_t o;
    if (rw.src < 0) {
      const uint32_t pv = f2bf(pad);
      o = (u32x4_t){pv | (pv << 16), pv | (pv << 16), pv | (pv << 16), pv | (pv << 16)};
    } else {
      float acc[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) acc[k] = 0.f;
      const int L = s_len[g], st = s_start[g];
      for (int j0 = 0; j0 < L; j0 += 8) {
        u32x4_t q[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int j = j0 + u, i = st + j;
          q[u] = (u32x4_t){0u, 0u, 0u, 0u};
          if (j < L) {
            if (i < DD_NMAX) {
              const int k = s_k[i];
              if (k >= 0)
                q[u] = s_u[k][l8];
              else if (k <= -2)
                q[u] = *(const u32x4_t*)(tab + (int64_t)s_key[-2 - k] * EMB_DIM + l8 * 8);
            } else {  // past the staged positions: straight from the arena and the table
              const int64_t pos = s_id0[g] + j;
              const int id = (pos >= 0 && pos < ids_len) ? ids[pos] : -1;
              if ((uint64_t)(int64_t)id < (uint64_t)table_rows)
                q[u] = *(const u32x4_t*)(tab + (int64_t)id * EMB_DIM + l8 * 8);
              else
                *err = 1;
            }
          }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (j0 + u < L) {
            acc[0] += bf2f(q[u].x & 0xffffu); acc[1] += bf2f(q[u].x >> 16);
            acc[2] += bf2f(q[u].y & 0xffffu); acc[3] += bf2f(q[u].y >> 16);
            acc[4] += bf2f(q[u].z & 0xffffu); acc[5] += bf2f(q[u].z >> 16);
            acc[6] += bf2f(q[u].w & 0xffffu); acc[7] += bf2f(q[u].w >> 16);
          }
        }
      }
      o.x = pack2(acc[0], acc[1]);
      o.y = pack2(acc[2], acc[3]);
      o.z = pack2(acc[4], acc[5]);
      o.w = pack2(acc[6], acc[7]);
    }
    *(u32x4_t*)(X + (int64_t)(r0 + g) * ldx + t * EMB_DIM + l8 * 8) = o;
  }
  // the workgroups of table 0 also write the rows' dense features and zero tails
  if (t == 0) {
    const int demb = n_tables * EMB_DIM;
    for (int i = 0; i < DD_ROWS && r0 + i < n_rows; ++i) {
      const rb_k_row rw = rows[r0 + i];
      bf16_t* xr = X + (int64_t)(r0 + i) * ldx;
      for (int c = demb + tid; c < ldx; c += DD_NT) {
        const int d = c - demb;
        xr[c] = d < n_dense ? f2bf(rw.src < 0 ? pad : dense[rw.src + d]) : (bf16_t)0;
      }
    }
  }
}

// ---------------------------------------------------------------- GEMM (bf16 and fp32)

// value of v in lane l ^ 2 / l ^ 1 of the same quad (DPP quad permutations:
// plain VALU moves, no LDS traffic)
__device__ __forceinline__ float quad_xor2(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, false));  // [2,3,0,1]
}
__device__ __forceinline__ float quad_xor1(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, false));  // [1,0,3,2]
}

// 4 x 4 transpose across the four lanes of a quad: lane 4q + i holding x[k] =
// element (k, i) ends up holding x[j] = element (i, j), where element (k, c)
// is the value lane 4q + c held in x[k]. Two exchange rounds (lane xor 2, then
// lane xor 1), each sending two values and keeping two, with selects only.
__device__ __forceinline__ void quad_transpose4(float (&x)[4], int lane) {
  const bool b1 = lane & 2, b0 = lane & 1;
  float r0 = quad_xor2(b1 ? x[0] : x[2]), r1 = quad_xor2(b1 ? x[1] : x[3]);
  const float y0 = b1 ? r0 : x[0], y1 = b1 ? r1 : x[1], y2 = b1 ? x[2] : r0, y3 = b1 ? x[3] : r1;
  r0 = quad_xor1(b0 ? y0 : y1);
  r1 = quad_xor1(b0 ? y2 : y3);
  x[0] = b0 ? r0 : y0;
  x[1] = b0 ? y1 : r0;
  x[2] = b0 ? r1 : y2;
  x[3] = b0 ? y3 : r1;
}

// two floats rounded to bf16 (round to nearest even, v_cvt_pk_bf16_f32),
// the first in the low half
__device__ __forceinline__ uint32_t pack2_rne(float a, float b) {
  typedef __bf16 bf16x2_hw __attribute__((ext_vector_type(2)));
  typedef float float2_hw __attribute__((ext_vector_type(2)));
  const float2_hw f = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_hw));
}

// s_waitcnt vmcnt(N) lgkmcnt(0) (gfx9 encoding: vmcnt[3:0], expcnt[6:4],
// lgkmcnt[11:8], vmcnt[5:4] in bits 15:14): at most N vector memory
// operations of this wave in flight and every LDS read of it returned.
template <int N>
__device__ __forceinline__ void wait_vmcnt_lds() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}

template <int I>
using ic = std::integral_constant<int, I>;

// f(ic<0>{}), f(ic<1>{}), ..., f(ic<N - 1>{}), unrolled at compile time
template <int... I, class F>
__device__ __forceinline__ void for_each_ic(std::integer_sequence<int, I...>, F&& f) {
  (f(ic<I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  for_each_ic(std::make_integer_sequence<int, N>{}, f);
}

// LDS byte address of a __shared__ object.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// Buffer resource (gfx9 layout: base address, stride 0, no range limit) for
// a wave-uniform base address.
__device__ __forceinline__ i32x4_t buffer_rsrc(const void* base) {
  const uint64_t p = (uint64_t)(uintptr_t)base;
  i32x4_t r;
  r.x = __builtin_amdgcn_readfirstlane((int)(uint32_t)p);
  r.y = __builtin_amdgcn_readfirstlane((int)((uint32_t)(p >> 32) & 0xffffu));
  r.z = -1;
  r.w = 0x00020000;
  return r;
}

// One 16-byte-per-lane buffer -> LDS load (buffer_load_dwordx4 ... lds) of the
// bytes at base + voff + soff: lane l's 16 bytes land at LDS byte lds + 16 l.
// Issued as inline assembly so that the compiler does not add its own
// conservative waits for it: the kernel waits with explicit vmcnt counts and
// a barrier before the data is read.
__device__ __forceinline__ void buffer_to_lds(i32x4_t rsrc, uint32_t voff, uint32_t soff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds" ::"s"(lds), "v"(voff), "s"(rsrc),
               "s"(soff)
               : "memory", "m0");
}

// Y = act(X W^T + b): X [M, K] and W [N, K] of element type TI (bf16 or
// fp32), K contiguous; fp32 accumulation with v_mfma_f32_32x32x16_bf16 or
// v_mfma_f32_32x32x2f32.
//
// Workgroup tile BM x BN, k-step of RB bytes per row (64 or 128: 32 or 64
// bf16, 16 or 32 fp32), NT/64 waves each owning a WM x WN sub-tile
// ((WM/32) x (WN/32) accumulators). Operand tiles go straight from global
// memory into a ring of S >= 2 LDS stages (global_load_lds: each wave load
// instruction fills 1 KB of consecutive LDS rows; no register staging).
// K-step kt reads stage kt % S while the stage of k-step kt - 1 is refilled
// with k-step kt - 1 + S, its loads spread one every few MFMAs over the step
// (over its first half when S = 2, where that refill is the next k-step):
// issued back to back they stall the wave on the texture path with no MFMA in
// flight. A sub-step covers 32 bytes of every row (16 bf16 or 8 fp32 k values)
// and its MFMAs have the next sub-step's fragment reads between them. In the
// last sub-step, after half of its MFMAs (three quarters with S = 2), the wave
// waits for its loads of the next k-step and for its LDS reads, and all waves
// meet at one barrier: the next stage has landed and nobody reads the current
// one again. The rest of the sub-step then runs with the next k-step's first
// fragment reads between the MFMAs. The order of MFMAs, LDS reads and loads
// within a step is fixed with scheduling barriers.
//
// A fragment is 16 bytes of one row: lane l holds row l % 32 and chunk
// 2 kk + l / 32 of sub-step kk. bf16: one 32x32x16 MFMA per accumulator and
// sub-step. fp32: chunk c holds k = 4c .. 4c + 3, and MFMA t (t = 0..3) of the
// sub-step takes dword t, so it adds the products of k = 8 kk + t (lanes
// 0..31) and k = 8 kk + 4 + t (lanes 32..63); the MFMAs of a sub-step run
// t-major over the accumulators, so two MFMAs into one accumulator are NM
// instructions apart.
//
// LDS rows hold RB/16 16-byte chunks; chunk c of row r sits at chunk
// c ^ ((r / (16 / (RB/16))) % (RB/16)), so the 16 rows one fragment read
// serves per LDS cycle hit 16 distinct bank groups (64 banks).
//
// Every tile shape, k-step, stage count and tile order accumulates each output
// element in the same k order with the same instructions, so results do not
// depend on them, nor on which rows share a tile.
//
// skip_rows (sequence layout, slot e owning rows [e skip_T, (e + 1) skip_T),
// skip_T a multiple of BM): a workgroup whose rows are all padding tokens
// (at or past its slot's length, or in a padding slot) returns at once.
constexpr int G16_KALIGN = 64;  // K multiple the bf16 entry point accepts
constexpr int G32_KALIGN = 32;  // K multiple the fp32 entry point accepts
constexpr int G32_BM = 64;      // fp32 tile height (the padding-token skip granularity)

// A narrow head applied in the epilogue instead of storing the layer's
// output (HEAD >= 0, the head's activation): the layer's bf16 outputs of
// the tile (all N = BN columns of its rows) go to LDS, and row r's head
// output act(w . y_r + b) is written to out[rows[r].out] when that is >= 0.
struct HeadArgs {
  const rb_k_row* rows;
  const bf16_t* w;  // BN bf16 weights, 16-byte aligned
  float b;
  float* out;
};

// fp32 outputs written through a row map instead of to Y (rows != nullptr):
// row r's first d_out columns go to out[rows[r].out ...] when that is >= 0
// (the merged run's split fused into its last layer); padding rows and
// columns past d_out are dropped.
struct OutMap {
  const rb_k_row* rows;
  float* out;
  int d_out;
};

template <typename TI, int BM, int BN, int WM, int WN, int NT, int RB, int S, int ORDER, int ACT, bool OUT_F32,
          bool PERSIST, int HEAD = -1>
__device__ __forceinline__ void gemm_mfma(const TI* __restrict__ X, int ldx, const TI* __restrict__ W, int ldw,
                                          const float* __restrict__ bias, void* __restrict__ Y, int ldy, int M,
                                          int N, int K, const rb_k_row* __restrict__ skip_rows, int skip_T,
                                          const HeadArgs ha = HeadArgs{}, const OutMap om = OutMap{}) {
  constexpr bool F32 = sizeof(TI) == 4;
  constexpr int ES = sizeof(TI);  // bytes per element
  constexpr int BK = RB / ES;     // k values per k-step
  constexpr int NW = NT / 64;
  static_assert((BM / WM) * (BN / WN) == NW, "one wave per sub-tile");
  static_assert(RB == 64 || RB == 128, "k-step of 64 or 128 bytes per row");
  static_assert(S >= 2 && S <= 4, "2..4 stages");
  constexpr int CPR = RB / 16;   // 16-byte chunks per LDS row
  constexpr int RPI = 64 / CPR;  // rows filled per wave load instruction
  constexpr int SWZ = 16 / CPR;  // rows sharing one swizzle pattern
  constexpr int EPC = 16 / ES;   // elements per chunk
  constexpr int TM = WM / 32, TN = WN / 32;
  static_assert(TM % 2 == 0 || F32, "the last sub-step splits the A fragments in halves");
  constexpr int SA = BM / RPI / NW, SB = BN / RPI / NW;  // load instructions per wave per stage
  static_assert(SA * NW * RPI == BM && SB * NW * RPI == BN, "loads cover the tile");
  constexpr int OPS = SA + SB;
  constexpr int KK = RB / 32;    // MFMA sub-steps per k-step
  constexpr int NM = TM * TN;    // accumulators
  constexpr int MPF = F32 ? 4 : 1;  // MFMAs per accumulator and sub-step
  constexpr int NU = NM * MPF;   // MFMAs per sub-step
  constexpr int NR = TM + TN;    // fragment reads per sub-step
  // the last sub-step's MFMAs before the barrier: half of them, three quarters
  // with two stages (more time for the loads of the next k-step to land)
  constexpr int UB = S == 2 ? NU * 3 / 4 : NU / 2;
  constexpr int PRE = (KK - 1) * NU + UB;  // MFMAs of a step before its barrier
  // MFMA slots the refill loads are spread over: with two stages the stage
  // refilled during a step is the one the next step reads, so its loads go in
  // the first half of the step to land before the barrier
  constexpr int LPOS = S == 2 ? PRE / 2 : PRE;
  // fragment read slot -> fragment (A fragments q < TM, then B). With two
  // stages (bf16) in the order the next sub-step's MFMAs consume them (A0, B0
  // .. B(TN-1), A1 .. A(TM-1)), so the fragment needed first is read first;
  // otherwise A0 .. A(TM-1), B0 .. B(TN-1).
  auto qmap = [](auto sc) {
    constexpr int q = decltype(sc)::value;
    if constexpr (S != 2 || F32 || q == 0)
      return ic<q>{};
    else if constexpr (q <= TN)
      return ic<TM + q - 1>{};
    else
      return ic<q - TN>{};
  };
  __shared__ u32x4_t sA[S][BM * CPR];
  __shared__ u32x4_t sB[S][BN * CPR];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid / (BN / WN), wn = wid % (BN / WN);
  const int tiles_n = N / BN;
  const int ntiles = ((M + BM - 1) / BM) * tiles_n;
  // v: this workgroup's index in the tile sequence (blockIdx.x, then + gridDim.x
  // per tile when persistent; gridDim.x is a multiple of 8, so v % 8 stays the
  // XCD the workgroup runs on)
  int v = blockIdx.x;
  auto tile_origin = [&](int vv, int& m0_, int& n0_) {
    const int tile = ORDER ? xcd_tile(vv, ntiles) : vv;
    const int bm = tile / tiles_n;
    m0_ = bm * BM;
    n0_ = (tile - bm * tiles_n) * BN;
  };
  int m0, n0;
  tile_origin(v, m0, n0);
  if (skip_rows) {  // uniform per workgroup
    const int e = m0 / skip_T;
    const rb_k_row rw = skip_rows[e];
    if (rw.src < 0 || m0 - e * skip_T >= rw.aux) return;
  }

  // lane l of a load instruction fills LDS row l / CPR (of its RPI), chunk l % CPR
  const int lr = lane / CPR, lc = lane % CPR;
  // byte offsets from the tile's first row (buffer resources based there; the
  // k-step's byte offset goes in the scalar offset)
  auto a_offsets = [&](int m0_, uint32_t (&va_)[SA]) {
#pragma unroll
    for (int i = 0; i < SA; ++i) {
      const int row = (wid * SA + i) * RPI + lr;
      const int ra = min(row, M - 1 - m0_);  // rows past M are computed on a copy and never stored
      va_[i] = (uint32_t)(ra * ldx + (lc ^ ((row / SWZ) % CPR)) * EPC) * (uint32_t)ES;
    }
  };
  i32x4_t rA = buffer_rsrc(X + (int64_t)m0 * ldx), rB = buffer_rsrc(W + (int64_t)n0 * ldw);
  uint32_t va[SA], vb[SB];
  a_offsets(m0, va);
#pragma unroll
  for (int i = 0; i < SB; ++i) {
    const int row = (wid * SB + i) * RPI + lr;
    vb[i] = (uint32_t)(row * ldw + (lc ^ ((row / SWZ) % CPR)) * EPC) * (uint32_t)ES;
  }
  // persistent: the next tile's origin, resources and A offsets (a copy of the
  // current tile's when there is none)
  int m0n = m0, n0n = n0;
  bool has_next = false;
  i32x4_t rAn = rA, rBn = rB;
  uint32_t van[SA];
#pragma unroll
  for (int i = 0; i < SA; ++i) van[i] = va[i];
  auto next_tile = [&]() {
    has_next = v + (int)gridDim.x < ntiles;
    if (has_next) {
      tile_origin(v + (int)gridDim.x, m0n, n0n);
      rAn = buffer_rsrc(X + (int64_t)m0n * ldx);
      rBn = buffer_rsrc(W + (int64_t)n0n * ldw);
      a_offsets(m0n, van);
    } else {
      m0n = m0;
      n0n = n0;
      rAn = rA;
      rBn = rB;
#pragma unroll
      for (int i = 0; i < SA; ++i) van[i] = va[i];
    }
  };
  if constexpr (PERSIST) next_tile();

  floatx16_t acc[TM][TN];
  auto zero_acc = [&]() {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  };
  zero_acc();

  const int nk = K / BK;
  // load instruction o (A rows for o < SA, then B rows) of k-step kt into
  // stage st. K-steps past the end reload the last one into a stage that is
  // never read again, so every step runs the same branch-free code; when
  // persistent, they are the next tile's first k-steps instead (the load stream
  // runs on across tiles, so the next tile's operands are in flight during this
  // tile's last steps and epilogue).
  auto issue_one = [&](int kt, auto stc, auto oc) {
    constexpr int st = decltype(stc)::value, o = decltype(oc)::value;
    if constexpr (PERSIST) {
      const bool nx = kt >= nk;  // uniform
      const uint32_t kb = (uint32_t)((nx ? (has_next ? kt - nk : nk - 1) : kt) * RB);
      if constexpr (o < SA)
        buffer_to_lds(nx ? rAn : rA, nx ? van[o] : va[o], kb, lds_addr(&sA[st][0]) + (wid * SA + o) * 1024);
      else
        buffer_to_lds(nx ? rBn : rB, vb[o - SA], kb, lds_addr(&sB[st][0]) + (wid * SB + o - SA) * 1024);
    } else {
      const uint32_t kb = (uint32_t)(min(kt, nk - 1) * RB);
      if constexpr (o < SA)
        buffer_to_lds(rA, va[o], kb, lds_addr(&sA[st][0]) + (wid * SA + o) * 1024);
      else
        buffer_to_lds(rB, vb[o - SA], kb, lds_addr(&sB[st][0]) + (wid * SB + o - SA) * 1024);
    }
  };
  u32x4_t fa[2][TM], fb[2][TN];
  // fragment read q (A fragment q for q < TM, then B) of sub-step kk of stage st
  auto read_one = [&](auto stc, int kk, auto qc, auto bufc) {
    constexpr int st = decltype(stc)::value, q = decltype(qc)::value, bf = decltype(bufc)::value;
    // lane l holds row l % 32, chunk 2 kk + l / 32
    const int ch = kk * 2 + (lane >> 5);
    if constexpr (q < TM) {
      const int r = wm * WM + q * 32 + (lane & 31);
      fa[bf][q] = sA[st][r * CPR + (ch ^ ((r / SWZ) % CPR))];
    } else {
      const int r = wn * WN + (q - TM) * 32 + (lane & 31);
      fb[bf][q - TM] = sB[st][r * CPR + (ch ^ ((r / SWZ) % CPR))];
    }
  };
  // k-step kt: stage stc, next stage nstc, refilled stage rstc (k-step kt - 1's)
  auto step = [&](int kt, auto stc, auto nstc, auto rstc) {
    static_for<KK>([&](auto kkc) {
      constexpr int kk = decltype(kkc)::value;
      constexpr bool last = kk == KK - 1;
      constexpr int cur = kk & 1, nxt = (kk + 1) & 1;
      static_for<NU>([&](auto uc) {
        constexpr int u = decltype(uc)::value;
        constexpr int m = u % NM, t = u / NM;
        if constexpr (last && u == UB) {
          wait_vmcnt_lds<(S - 2) * OPS>();
          lds_barrier();
        }
        if constexpr (F32)
          acc[m / TN][m % TN] = __builtin_amdgcn_mfma_f32_32x32x2f32(
              __uint_as_float(fa[cur][m / TN][t]), __uint_as_float(fb[cur][m % TN][t]), acc[m / TN][m % TN], 0, 0, 0);
        else
          acc[m / TN][m % TN] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8_t, fa[cur][m / TN]), __builtin_bit_cast(bf16x8_t, fb[cur][m % TN]),
              acc[m / TN][m % TN], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
        static_for<NR>([&](auto qc) {
          constexpr int q = decltype(qc)::value;
          if constexpr (!last) {
            if constexpr (q * NU / NR == u) read_one(stc, kk + 1, qmap(qc), ic<nxt>{});
          } else if constexpr (u >= UB) {
            if constexpr (UB + q * (NU - UB) / NR == u) read_one(nstc, 0, qmap(qc), ic<0>{});
          }
        });
        constexpr int pos = kk * NU + u;
        static_for<OPS>([&](auto oc) {
          constexpr int o = decltype(oc)::value;
          if constexpr (o * LPOS / OPS == pos) issue_one(kt - 1 + S, rstc, oc);
        });
        __builtin_amdgcn_sched_barrier(0);
      });
    });
  };
  static_for<S - 1>([&](auto sc) { static_for<OPS>([&](auto oc) { issue_one(decltype(sc)::value, sc, oc); }); });
  wait_vmcnt_lds<(S - 2) * OPS>();
  lds_barrier();
  static_for<NR>([&](auto qc) { read_one(ic<0>{}, 0, qmap(qc), ic<0>{}); });
  auto group = [&](int kt) {  // S k-steps from a multiple of S
    step(kt, ic<0>{}, ic<1>{}, ic<S - 1>{});
    step(kt + 1, ic<1>{}, ic<2 % S>{}, ic<0>{});
    if constexpr (S > 2) step(kt + 2, ic<2 % S>{}, ic<3 % S>{}, ic<1>{});
    if constexpr (S > 3) step(kt + 3, ic<3>{}, ic<0>{}, ic<2>{});
  };

  // accumulator (i, j) register r of lane l holds row 8*(r/4) + 4*(l/32) + r%4,
  // column l%32 of its 32 x 32 block. Bias and activation are applied per
  // column; then each group of four registers (four consecutive rows) is
  // transposed across the four lanes of a quad, so that a lane holds four
  // consecutive columns of one row and stores them at once (8 bytes bf16, 16
  // bytes fp32) instead of four single elements.
  auto epilogue = [&]() {
  // with an output row map: the output offsets of this lane's rows, loaded
  // all at once before any is needed
  const bool mapped = OUT_F32 && om.rows != nullptr;  // uniform
  int64_t ro[TM][4];
  if (mapped) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int r = m0 + wm * WM + i * 32 + 8 * g + 4 * (lane >> 5) + (lane & 3);
        ro[i][g] = r < M ? om.rows[r].out : -1;
      }
  }
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const float bb = bias[n0 + wn * WN + j * 32 + (lane & 31)];
    const int colq = n0 + wn * WN + j * 32 + (lane & 28);  // first column of this lane's quad
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float q[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) q[k] = act_fn<ACT>(acc[i][j][4 * g + k] + bb);
        quad_transpose4(q, lane);
        const int row = m0 + wm * WM + i * 32 + 8 * g + 4 * (lane >> 5) + (lane & 3);
        // streaming (nontemporal) stores: the whole chip writes its tiles'
        // outputs at about the same time, and these drain faster than
        // stores that allocate in L2
        if constexpr (OUT_F32) {
          if (mapped) {
            const int64_t o = ro[i][g];
            if (o >= 0) {
              float* dst = om.out + o + colq;
              if (colq + 3 < om.d_out && ((uintptr_t)dst & 15) == 0) {
                const f32x4_t v = {q[0], q[1], q[2], q[3]};
                __builtin_nontemporal_store(v, (f32x4_t*)dst);
              } else {
#pragma unroll
                for (int k = 0; k < 4; ++k)
                  if (colq + k < om.d_out) dst[k] = q[k];
              }
            }
            continue;
          }
        }
        if (row < M) {
          if (OUT_F32) {
            const f32x4_t o = {q[0], q[1], q[2], q[3]};
            __builtin_nontemporal_store(o, (f32x4_t*)((float*)Y + (int64_t)row * ldy + colq));
          } else {
            const u32x2_t o = {pack2_rne(q[0], q[1]), pack2_rne(q[2], q[3])};
            __builtin_nontemporal_store(o, (u32x2_t*)((bf16_t*)Y + (int64_t)row * ldy + colq));
          }
        }
      }
  }
  };

  // The head instead of the store: the tile's outputs, rounded to bf16 exactly
  // as the store would round them, into LDS rows of HLD bytes (over the
  // operand stages, once every wave is done with them); then 16 lanes per row
  // sum w . y in the order of k_head (lane l: elements 8 l .. 8 l + 7 of every
  // 128, then a 16-lane butterfly), so the results equal the separate layer and
  // head bit for bit.
  auto head_epilogue = [&]() {
    if constexpr (HEAD >= 0) {
    constexpr int RPP = NT / 16;  // rows per pass of the head (16 lanes each)
    static_assert(!F32 && !OUT_F32 && BN == 256 && BM % RPP == 0, "bf16 layer of 256 outputs");
    constexpr int HLD = BN * 2 + 16;
    static_assert(BM * HLD <= S * BN * CPR * 16, "the output tile fits over the B stages");
    unsigned char* hb = (unsigned char*)&sB[0][0];
    // the output offsets of this thread's rows and its head weights, loaded
    // before the tile goes to LDS so that their latency overlaps it
    const int l = tid & 15;
    int64_t outs[BM / RPP];
#pragma unroll
    for (int p = 0; p < BM / RPP; ++p) {
      const int r = m0 + p * RPP + (tid >> 4);
      outs[p] = r < M ? ha.rows[r].out : -1;
    }
    const u32x4_t w0 = *(const u32x4_t*)(ha.w + l * 8), w1 = *(const u32x4_t*)(ha.w + 128 + l * 8);
    __syncthreads();
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const float bb = bias[n0 + wn * WN + j * 32 + (lane & 31)];
      const int colq = wn * WN + j * 32 + (lane & 28);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float q[4];
#pragma unroll
          for (int k = 0; k < 4; ++k) q[k] = act_fn<ACT>(acc[i][j][4 * g + k] + bb);
          quad_transpose4(q, lane);
          const int rl = wm * WM + i * 32 + 8 * g + 4 * (lane >> 5) + (lane & 3);
          const u32x2_t o = {pack2_rne(q[0], q[1]), pack2_rne(q[2], q[3])};
          *(u32x2_t*)(hb + rl * HLD + colq * 2) = o;
        }
    }
    __syncthreads();
#pragma unroll
    for (int p = 0; p < BM / RPP; ++p) {
      const int rl = p * RPP + (tid >> 4);
      float sum = 0.f;
      const int64_t o = outs[p];
      {
        if (o >= 0) {
#pragma unroll
          for (int c = 0; c < 2; ++c) {
            const u32x4_t hv = *(const u32x4_t*)(hb + rl * HLD + (c * 128 + l * 8) * 2), wv = c ? w1 : w0;
            sum += bf2f(hv.x & 0xffffu) * bf2f(wv.x & 0xffffu);
            sum += bf2f(hv.x >> 16) * bf2f(wv.x >> 16);
            sum += bf2f(hv.y & 0xffffu) * bf2f(wv.y & 0xffffu);
            sum += bf2f(hv.y >> 16) * bf2f(wv.y >> 16);
            sum += bf2f(hv.z & 0xffffu) * bf2f(wv.z & 0xffffu);
            sum += bf2f(hv.z >> 16) * bf2f(wv.z >> 16);
            sum += bf2f(hv.w & 0xffffu) * bf2f(wv.w & 0xffffu);
            sum += bf2f(hv.w >> 16) * bf2f(wv.w >> 16);
          }
        }
      }
      sum += __shfl_xor(sum, 1);
      sum += __shfl_xor(sum, 2);
      sum += __shfl_xor(sum, 4);
      sum += __shfl_xor(sum, 8);
      if (l == 0 && o >= 0) ha.out[o] = act_fn<HEAD>(sum + ha.b);
    }
    }
  };

  if constexpr (PERSIST) {
    // K a multiple of S k-steps (so every tile starts at stage 0) and at least
    // S k-steps (so the loads of a tile's last steps reach only the next tile)
    for (;;) {
      for (int kt = 0; kt < nk; kt += S) group(kt);
      epilogue();
      if (!has_next) break;
      v += gridDim.x;
      m0 = m0n;
      n0 = n0n;
      rA = rAn;
      rB = rBn;
#pragma unroll
      for (int i = 0; i < SA; ++i) va[i] = van[i];
      next_tile();
      zero_acc();
    }
    // no load into LDS may still be in flight when the wave ends
    wait_vmcnt_lds<0>();
  } else {
    int kt = 0;
    for (; kt + S <= nk; kt += S) group(kt);
    if (kt < nk) step(kt, ic<0>{}, ic<1>{}, ic<S - 1>{});
    if (kt + 1 < nk) step(kt + 1, ic<1>{}, ic<2 % S>{}, ic<0>{});
    if constexpr (S > 3)
      if (kt + 2 < nk) step(kt + 2, ic<2 % S>{}, ic<3 % S>{}, ic<1>{});
    // no load into LDS may still be in flight when the wave ends
    wait_vmcnt_lds<0>();
    if constexpr (HEAD >= 0)
      head_epilogue();
    else
      epilogue();
  }
}

// The two operand types as separately named kernels (so that traces and
// counters tell them apart).
template <int BM, int BN, int WM, int WN, int NT, int RB, int S, int ORDER, int ACT, bool OUT_F32, bool PERSIST>
__global__ __launch_bounds__(NT) void k_gemm_bf16(const bf16_t* __restrict__ X, int ldx,
                                                  const bf16_t* __restrict__ W, int ldw,
                                                  const float* __restrict__ bias, void* __restrict__ Y, int ldy,
                                                  int M, int N, int K, OutMap om) {
  gemm_mfma<bf16_t, BM, BN, WM, WN, NT, RB, S, ORDER, ACT, OUT_F32, PERSIST>(X, ldx, W, ldw, bias, Y, ldy, M, N, K,
                                                                            nullptr, 0, HeadArgs{}, om);
}
// A bf16 layer of 256 outputs with a narrow head in its epilogue (HEAD: the
// head's activation); the layer's outputs never leave the workgroup.
template <int BM, int BN, int WM, int WN, int NT, int RB, int S, int ORDER, int ACT, int HEAD>
__global__ __launch_bounds__(NT) void k_gemm_head(const bf16_t* __restrict__ X, int ldx,
                                                  const bf16_t* __restrict__ W, int ldw,
                                                  const float* __restrict__ bias, int M, int K, HeadArgs ha) {
  gemm_mfma<bf16_t, BM, BN, WM, WN, NT, RB, S, ORDER, ACT, false, false, HEAD>(X, ldx, W, ldw, bias, nullptr, BN, M,
                                                                             BN, K, nullptr, 0, ha);
}
template <int BM, int BN, int WM, int WN, int NT, int RB, int S, int ORDER, int ACT>
__global__ __launch_bounds__(NT) void k_gemm_f32(const float* __restrict__ X, int ldx, const float* __restrict__ W,
                                                 int ldw, const float* __restrict__ bias, void* __restrict__ Y,
                                                 int ldy, int M, int N, int K,
                                                 const rb_k_row* __restrict__ skip_rows, int skip_T, OutMap om) {
  gemm_mfma<float, BM, BN, WM, WN, NT, RB, S, ORDER, ACT, true, false>(X, ldx, W, ldw, bias, Y, ldy, M, N, K,
                                                                       skip_rows, skip_T, HeadArgs{}, om);
}

// ---------------------------------------------------------------- heads and split

// 16 lanes per row (16 rows per workgroup): a K-long dot product, each lane
// taking 8 consecutive elements of every 128 with 16-byte loads (or every
// 16th element when rows are not 16-byte aligned), a 16-lane butterfly, bias,
// activation, and the store into the request's output row (one wave per row
// with 2-byte loads measured 1.5x slower on 256-wide rows).
template <int ACT>
__global__ __launch_bounds__(256) void k_head(const rb_k_row* __restrict__ rows, int n,
                                              const bf16_t* __restrict__ H, int ldh,
                                              const bf16_t* __restrict__ w, float b, int K, int vec,
                                              float* __restrict__ out) {
  const int r = blockIdx.x * 16 + (threadIdx.x >> 4), l = threadIdx.x & 15;
  float s = 0.f;
  int64_t o = -1;
  if (r < n) {
    o = rows[r].out;
    if (o >= 0) {
      const bf16_t* h = H + (int64_t)r * ldh;
      if (vec) {
        for (int k = l * 8; k < K; k += 128) {
          const u32x4_t hv = *(const u32x4_t*)(h + k), wv = *(const u32x4_t*)(w + k);
          s += bf2f(hv.x & 0xffffu) * bf2f(wv.x & 0xffffu);
          s += bf2f(hv.x >> 16) * bf2f(wv.x >> 16);
          s += bf2f(hv.y & 0xffffu) * bf2f(wv.y & 0xffffu);
          s += bf2f(hv.y >> 16) * bf2f(wv.y >> 16);
          s += bf2f(hv.z & 0xffffu) * bf2f(wv.z & 0xffffu);
          s += bf2f(hv.z >> 16) * bf2f(wv.z >> 16);
          s += bf2f(hv.w & 0xffffu) * bf2f(wv.w & 0xffffu);
          s += bf2f(hv.w >> 16) * bf2f(wv.w >> 16);
        }
      } else {
        for (int k = l; k < K; k += 16) s += bf2f(h[k]) * bf2f(w[k]);
      }
    }
  }
  // 16-lane sum: every lane of the wave takes part in the exchanges
  s += __shfl_xor(s, 1);
  s += __shfl_xor(s, 2);
  s += __shfl_xor(s, 4);
  s += __shfl_xor(s, 8);
  if (l == 0 && o >= 0) out[o] = act_fn<ACT>(s + b);
}

// ---------------------------------------------------------------- fused MLP tail

// The last two hidden layers (ReLU, N2 = 512 then N3 = 256 outputs) and the
// narrow head of a bf16 model, fused per block of MT_BM rows: the first layer's
// k-steps stream H1 rows and W2 rows through two LDS stages; its outputs
// (bias, ReLU, bf16) stay in LDS as the second layer's input while W3 streams
// through two more stages; the second layer's outputs (bias, ReLU, bf16) go to
// LDS and the head reads them there. Each output is accumulated in the same k
// order with the same 32x32x16 bf16 MFMA as k_gemm_bf16, rounded the same way,
// and the head sums exactly as k_head does (16 lanes per row, 8 consecutive
// elements of every 128 per lane, then a 16-lane butterfly), so the results
// are bit-identical to running the two layers and the head separately; only
// the two hidden layers' round trips through memory and two launches go away.
// 8 waves: 2 x 4 over the 128 x 512 tile of the first layer (64 x 128 each),
// 2 x 4 over the 128 x 256 tile of the second (64 x 64 each). Operand rows of
// 64 bytes per k-step sit in LDS with their four 16-byte chunks permuted by
// row, and the 1024-byte rows of the first layer's output with their 64 chunks
// permuted by row, so that a fragment read's 32 rows spread over the banks.
constexpr int MT_BM = 128, MT_NT = 512, MT_N2 = 512, MT_N3 = 256, MT_KS = 32;
constexpr int MT_A_BYTES = MT_BM * 64, MT_B_BYTES = MT_N2 * 64;           // one stage of the first layer
constexpr int MT_Y2 = 0;                                                // [MT_BM][MT_N2] bf16, 128 KB
constexpr int MT_W3 = MT_BM * MT_N2 * 2;                                // two stages of [MT_N3][64 B]
constexpr int MT_LDS = MT_W3 + 2 * MT_N3 * 64;                          // 160 KB
static_assert(2 * (MT_A_BYTES + MT_B_BYTES) <= MT_W3, "first-layer stages fit below the W3 stages");

__device__ __forceinline__ uint32_t mt_addr4(int row, int c) { return (uint32_t)(row * 64 + ((c ^ ((row >> 2) & 3)) << 4)); }
__device__ __forceinline__ uint32_t mt_addr_y2(int row, int c) { return (uint32_t)(row * 1024 + ((c ^ (row & 63)) << 4)); }

template <int ACT>
__global__ __launch_bounds__(MT_NT) void k_mlp_tail(const bf16_t* __restrict__ H1, int ldh1, int K2,
                                                    const bf16_t* __restrict__ W2, int ldw2,
                                                    const float* __restrict__ b2, const bf16_t* __restrict__ W3,
                                                    int ldw3, const float* __restrict__ b3,
                                                    const bf16_t* __restrict__ w4, float b4,
                                                    const rb_k_row* __restrict__ rows, int M,
                                                    float* __restrict__ out) {
  __shared__ __align__(16) unsigned char lds[MT_LDS];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wid >> 2, wn = wid & 3;
  const int m0 = blockIdx.x * MT_BM;
  const int lrow = tid >> 2, lc = tid & 3;  // the row (of 128) and chunk this thread loads
  // ---- first layer: Y2 = relu(H1 W2^T + b2) on rows [m0, m0 + 128)
  const bf16_t* a_src = H1 + (int64_t)(m0 + min(lrow, M - 1 - m0)) * ldh1 + lc * 8;  // rows past M: a copy
  // k-step operands go global -> registers -> LDS, loaded two k-steps ahead
  // into two register sets (the k loops are unrolled by two so that each set
  // stays in registers)
  struct Op1 {
    u32x4_t a, b[4];
  };
  auto load1 = [&](Op1& r, int kt) {
    const int k0 = kt * MT_KS;
    r.a = *(const u32x4_t*)(a_src + k0);
#pragma unroll
    for (int i = 0; i < 4; ++i) r.b[i] = *(const u32x4_t*)(W2 + (int64_t)(lrow + 128 * i) * ldw2 + k0 + lc * 8);
  };
  auto store1 = [&](const Op1& r, int st) {
    unsigned char* base = lds + st * (MT_A_BYTES + MT_B_BYTES);
    *(u32x4_t*)(base + mt_addr4(lrow, lc)) = r.a;
#pragma unroll
    for (int i = 0; i < 4; ++i) *(u32x4_t*)(base + MT_A_BYTES + mt_addr4(lrow + 128 * i, lc)) = r.b[i];
  };
  floatx16_t acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  auto mma1 = [&](int st) {
    const unsigned char* base = lds + st * (MT_A_BYTES + MT_B_BYTES);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int c = kk * 2 + (lane >> 5);
      u32x4_t fa[2], fb[4];
#pragma unroll
      for (int i = 0; i < 2; ++i) fa[i] = *(const u32x4_t*)(base + mt_addr4(wm * 64 + i * 32 + (lane & 31), c));
#pragma unroll
      for (int j = 0; j < 4; ++j)
        fb[j] = *(const u32x4_t*)(base + MT_A_BYTES + mt_addr4(wn * 128 + j * 32 + (lane & 31), c));
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, fa[i]),
                                                              __builtin_bit_cast(bf16x8_t, fb[j]), acc[i][j], 0, 0, 0);
    }
  };
  // k-step kt: load kt + 2 into the set kt held, multiply stage kt % 2, store
  // kt + 1 (loaded a k-step ago) into the other stage
  auto step1 = [&](int kt, int nk, Op1& mine, Op1& next) {
    if (kt + 2 < nk) load1(mine, kt + 2);
    mma1(kt & 1);
    if (kt + 1 < nk) store1(next, (kt + 1) & 1);
    __syncthreads();
  };
  const int nk = K2 / MT_KS;
  Op1 r0, r1;
  load1(r0, 0);
  if (nk > 1) load1(r1, 1);
  store1(r0, 0);
  __syncthreads();
  for (int kt = 0; kt < nk; kt += 2) {
    step1(kt, nk, r0, r1);
    if (kt + 1 < nk) step1(kt + 1, nk, r1, r0);
  }
  // W3's first two k-steps load while the first layer's outputs go to LDS
  struct Op2 {
    u32x4_t b[2];
  };
  auto load2 = [&](Op2& r, int kt) {
    const int k0 = kt * MT_KS;
#pragma unroll
    for (int i = 0; i < 2; ++i) r.b[i] = *(const u32x4_t*)(W3 + (int64_t)(lrow + 128 * i) * ldw3 + k0 + lc * 8);
  };
  auto store2 = [&](const Op2& r, int st) {
    unsigned char* base = lds + MT_W3 + st * (MT_N3 * 64);
#pragma unroll
    for (int i = 0; i < 2; ++i) *(u32x4_t*)(base + mt_addr4(lrow + 128 * i, lc)) = r.b[i];
  };
  Op2 w0, w1;
  load2(w0, 0);
  load2(w1, 1);
  // accumulator (i, j) register r of lane l: row 8 (r / 4) + 4 (l / 32) + r % 4,
  // column l % 32 of its 32 x 32 block; bias and ReLU per column, then each
  // group of four rows transposed across the quad so a lane holds four
  // consecutive columns of one row (as k_gemm_bf16's epilogue), rounded to bf16
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int col0 = wn * 128 + j * 32;
    const float bb = b2[col0 + (lane & 31)];
    const int colq = col0 + (lane & 28);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float q[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) q[k] = act_fn<RB_ACT_RELU>(acc[i][j][4 * g + k] + bb);
        quad_transpose4(q, lane);
        const int row = wm * 64 + i * 32 + 8 * g + 4 * (lane >> 5) + (lane & 3);
        const u32x2_t o = {pack2_rne(q[0], q[1]), pack2_rne(q[2], q[3])};
        *(u32x2_t*)(lds + MT_Y2 + mt_addr_y2(row, colq >> 3) + ((colq & 4) ? 8 : 0)) = o;
      }
  }
  store2(w0, 0);
  __syncthreads();
  // ---- second layer: Y3 = relu(Y2 W3^T + b3)
  floatx16_t acc3[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc3[i][j][r] = 0.f;
  auto mma2 = [&](int kt) {
    const unsigned char* base = lds + MT_W3 + (kt & 1) * (MT_N3 * 64);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const int c = kk * 2 + (lane >> 5);
      u32x4_t fa[2], fb[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int row = wm * 64 + i * 32 + (lane & 31);
        fa[i] = *(const u32x4_t*)(lds + MT_Y2 + mt_addr_y2(row, kt * 4 + c));
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) fb[j] = *(const u32x4_t*)(base + mt_addr4(wn * 64 + j * 32 + (lane & 31), c));
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc3[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, fa[i]),
                                                               __builtin_bit_cast(bf16x8_t, fb[j]), acc3[i][j], 0, 0, 0);
    }
  };
  constexpr int nk3 = MT_N2 / MT_KS;
  auto step2 = [&](int kt, Op2& mine, Op2& next) {
    if (kt + 2 < nk3) load2(mine, kt + 2);
    mma2(kt);
    if (kt + 1 < nk3) store2(next, (kt + 1) & 1);
    __syncthreads();
  };
  for (int kt = 0; kt < nk3; kt += 2) {
    step2(kt, w0, w1);
    step2(kt + 1, w1, w0);
  }
  // Y3 (bias, ReLU, bf16) to LDS, row-major [MT_BM][MT_N3] over the first
  // layer's outputs (no longer read)
  unsigned char* y3 = lds;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int col0 = wn * 64 + j * 32;
    const float bb = b3[col0 + (lane & 31)];
    const int colq = col0 + (lane & 28);
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float q[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) q[k] = act_fn<RB_ACT_RELU>(acc3[i][j][4 * g + k] + bb);
        quad_transpose4(q, lane);
        const int row = wm * 64 + i * 32 + 8 * g + 4 * (lane >> 5) + (lane & 3);
        const u32x2_t o = {pack2_rne(q[0], q[1]), pack2_rne(q[2], q[3])};
        *(u32x2_t*)(y3 + row * (MT_N3 * 2) + colq * 2) = o;
      }
  }
  __syncthreads();
  // ---- head, as k_head: 16 lanes per row, lane l taking elements
  // [8 l + 128 i, 8 l + 128 i + 8), then a 16-lane butterfly
  const int l16 = tid & 15;
#pragma unroll
  for (int pass = 0; pass < MT_BM / (MT_NT / 16); ++pass) {
    const int row = pass * (MT_NT / 16) + (tid >> 4);
    float s = 0.f;
    for (int k = l16 * 8; k < MT_N3; k += 128) {
      const u32x4_t hv = *(const u32x4_t*)(y3 + row * (MT_N3 * 2) + k * 2), wv = *(const u32x4_t*)(w4 + k);
      s += bf2f(hv.x & 0xffffu) * bf2f(wv.x & 0xffffu);
      s += bf2f(hv.x >> 16) * bf2f(wv.x >> 16);
      s += bf2f(hv.y & 0xffffu) * bf2f(wv.y & 0xffffu);
      s += bf2f(hv.y >> 16) * bf2f(wv.y >> 16);
      s += bf2f(hv.z & 0xffffu) * bf2f(wv.z & 0xffffu);
      s += bf2f(hv.z >> 16) * bf2f(wv.z >> 16);
      s += bf2f(hv.w & 0xffffu) * bf2f(wv.w & 0xffffu);
      s += bf2f(hv.w >> 16) * bf2f(wv.w >> 16);
    }
    s += __shfl_xor(s, 1);
    s += __shfl_xor(s, 2);
    s += __shfl_xor(s, 4);
    s += __shfl_xor(s, 8);
    if (l16 == 0 && m0 + row < M) {
      const int64_t o = rows[m0 + row].out;
      if (o >= 0) out[o] = act_fn<ACT>(s + b4);
    }
  }
}

constexpr int POOL_MAX_D = 1024, POOL_MAX_OUT = 16;

// One workgroup per sequence slot. Wave w sums the slot's real tokens
// [w L / 4, (w + 1) L / 4) (tokens past L are never read, so padding cannot
// reach the mean), each lane owning float4 columns and keeping four token
// loads in flight while adding them in token order; the four partial sums are
// added in wave order and divided by L (a fixed order, so the result depends
// on the sequence only). The block then computes the head logits with
// fixed-order reductions and thread 0 applies the softmax and writes the
// request's output row.
__global__ __launch_bounds__(256) void k_seqpool(const rb_k_row* __restrict__ rows, int n_seqs, int T,
                                                 int64_t packed_rows, const float* __restrict__ H, int ldh, int D,
                                                 const float* __restrict__ Wh,
                                                 const float* __restrict__ bh, int n_out, int act,
                                                 float* __restrict__ out) {
  const int r = blockIdx.x;
  const rb_k_row rw = rows[r];
  if (rw.out < 0) return;
  int L = (int)min(max(rw.aux, (int64_t)0), (int64_t)T);  // reads stay inside the slot
  // packed tokens: the sequence's rows [rows[r].lens, + L) of packed_rows
  if (packed_rows > 0 && (rw.lens < 0 || rw.lens + L > packed_rows)) L = 0;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  __shared__ float psum[4][POOL_MAX_D];
  __shared__ float pooled[POOL_MAX_D];
  __shared__ float part[4][POOL_MAX_OUT];
  const float* h = H + (packed_rows > 0 ? rw.lens : (int64_t)r * T) * ldh;
  const int t0 = (int)((int64_t)L * wid / 4), t1 = (int)((int64_t)L * (wid + 1) / 4);
  if ((D & 3) == 0 && (ldh & 3) == 0) {
    for (int c = lane * 4; c < D; c += 256) {
      float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
      int t = t0;
      for (; t + 4 <= t1; t += 4) {
        float4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = *(const float4*)(h + (int64_t)(t + u) * ldh + c);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          s.x += v[u].x; s.y += v[u].y; s.z += v[u].z; s.w += v[u].w;
        }
      }
      for (; t < t1; ++t) {
        const float4 v = *(const float4*)(h + (int64_t)t * ldh + c);
        s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
      }
      *(float4*)&psum[wid][c] = s;
    }
  } else {
    for (int c = lane; c < D; c += 64) {
      float s = 0.f;
      for (int t = t0; t < t1; ++t) s += h[(int64_t)t * ldh + c];
      psum[wid][c] = s;
    }
  }
  __syncthreads();
  const float inv = 1.f / (float)max(L, 1);
  for (int c = tid; c < D; c += 256) pooled[c] = (((psum[0][c] + psum[1][c]) + psum[2][c]) + psum[3][c]) * inv;
  __syncthreads();
  for (int j = 0; j < n_out; ++j) {
    float s = 0.f;
    for (int c = tid; c < D; c += 256) s += Wh[(int64_t)j * D + c] * pooled[c];
    s = wave_sum(s);
    if (lane == 0) part[wid][j] = s;
  }
  __syncthreads();
  if (tid == 0) {
    float z[POOL_MAX_OUT];
    float mx = -INFINITY;
    for (int j = 0; j < n_out; ++j) {
      z[j] = ((part[0][j] + part[1][j]) + (part[2][j] + part[3][j])) + bh[j];
      mx = fmaxf(mx, z[j]);
    }
    if (act == RB_ACT_SOFTMAX) {
      float den = 0.f;
      for (int j = 0; j < n_out; ++j) {
        z[j] = expf(z[j] - mx);
        den += z[j];
      }
      for (int j = 0; j < n_out; ++j) out[rw.out + j] = z[j] / den;
    } else {
      for (int j = 0; j < n_out; ++j) out[rw.out + j] = z[j];
    }
  }
}

// Split: TPR threads per row, 256 / TPR rows per workgroup. With V = 4 a row
// whose output offset is a multiple of 4 floats is copied with 16-byte loads
// and stores (Y rows always are; output rows of a mixed-width arena may not
// be, and those take the scalar path).
template <int V>
__global__ __launch_bounds__(256) void k_split(const rb_k_row* __restrict__ rows, int n, int tpr,
                                               const float* __restrict__ Y, int ldy, int d_out,
                                               float* __restrict__ out) {
  const int rpb = 256 / tpr;
  const int r = blockIdx.x * rpb + threadIdx.x / tpr;
  if (r >= n) return;
  const int64_t o = rows[r].out;
  if (o < 0) return;
  const float* y = Y + (int64_t)r * ldy;
  const int t = threadIdx.x % tpr;
  if (V == 4 && (o & 3) == 0) {
    for (int c = t * 4; c < d_out; c += tpr * 4) *(float4*)(out + o + c) = *(const float4*)(y + c);
  } else {
    for (int c = t; c < d_out; c += tpr) out[o + c] = y[c];
  }
}

inline rb_status launch_status() {
  return hipGetLastError() == hipSuccess ? RB_OK : RB_EDEVICE;
}

inline unsigned blocks_for(int64_t threads) { return (unsigned)((threads + 255) / 256); }

}  // namespace

namespace {

// PERSIST: a grid of at most `cap` workgroups (a multiple of 8), each taking
// every cap-th tile
template <typename TI, int BM, int BN, int WM, int WN, int NT, int RB, int S, int ORDER, bool PERSIST = false>
void launch_gemm(hipStream_t s, const TI* x, int ldx, const TI* w, int ldw, const float* b, void* Y, int ldy,
                 int M, int N, int K, int act, bool out_f32, const rb_k_row* skip_rows, int skip_T,
                 unsigned cap = 0, OutMap om = OutMap{}) {
  const unsigned tiles = (unsigned)(((M + BM - 1) / BM) * (N / BN));
  const unsigned g = PERSIST ? std::min(tiles, cap) : tiles;
  if constexpr (sizeof(TI) == 4) {
#define RB_G(A)                                                                                                     \
  hipLaunchKernelGGL((k_gemm_f32<BM, BN, WM, WN, NT, RB, S, ORDER, A>), dim3(g), dim3(NT), 0, s, x, ldx, w, ldw, b, \
                     Y, ldy, M, N, K, skip_rows, skip_T, om)
    if (act == RB_ACT_RELU) RB_G(RB_ACT_RELU);
    else if (act == RB_ACT_SIGMOID) RB_G(RB_ACT_SIGMOID);
    else RB_G(RB_ACT_NONE);
#undef RB_G
  } else {
#define RB_G(A, F)                                                                                             \
  hipLaunchKernelGGL((k_gemm_bf16<BM, BN, WM, WN, NT, RB, S, ORDER, A, F, PERSIST>), dim3(g), dim3(NT), 0, s, x, ldx, w, \
                     ldw, b, Y, ldy, M, N, K, om)
    if (out_f32) {
      if (act == RB_ACT_RELU) RB_G(RB_ACT_RELU, true);
      else if (act == RB_ACT_SIGMOID) RB_G(RB_ACT_SIGMOID, true);
      else RB_G(RB_ACT_NONE, true);
    } else {
      if (act == RB_ACT_RELU) RB_G(RB_ACT_RELU, false);
      else if (act == RB_ACT_SIGMOID) RB_G(RB_ACT_SIGMOID, false);
      else RB_G(RB_ACT_NONE, false);
    }
#undef RB_G
  }
}

// bf16 operands, k-step BK bf16 values
template <int BM, int BN, int WM, int WN, int NT, int BK, int S, int ORDER, bool PERSIST>
void launch_gemm_bf16(hipStream_t s, const bf16_t* x, int ldx, const bf16_t* w, int ldw, const float* b, void* Y,
                      int ldy, int M, int N, int K, int act, int out_f32, unsigned cap, OutMap om) {
  launch_gemm<bf16_t, BM, BN, WM, WN, NT, BK * 2, S, ORDER, PERSIST>(s, x, ldx, w, ldw, b, Y, ldy, M, N, K, act,
                                                                    out_f32 != 0, nullptr, 0, cap, om);
}

// compute units of the current device (cached per device)
unsigned device_cus() {
  static std::atomic<int> cus[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int c = cus[dev].load(std::memory_order_relaxed);
  if (c <= 0) {
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || c <= 0) c = 256;
    cus[dev].store(c, std::memory_order_relaxed);
  }
  return (unsigned)c;
}

}  // namespace

// ---------------------------------------------------------------- row map fill

namespace {
// Every entry of a row map set to padding (no input, no output).
__global__ __launch_bounds__(256) void k_fill_padding_rows(rb_k_row* __restrict__ rows, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) rows[i] = rb_k_row{-1, 0, -1, -1};
}
}  // namespace

// Runtime support (not part of the C ABI): a row map whose batches come from
// a caller's descriptors starts as padding, so that rows no valid batch
// covers are neither computed from nor returned.
void rb_fill_padding_rows(hipStream_t stream, rb_k_row* rows, int64_t n) {
  if (n > 0) hipLaunchKernelGGL(k_fill_padding_rows, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, rows, n);
}

// ---------------------------------------------------------------- static scratch

namespace {
// Work memory of the allocation-free launch-group entry point: one copy per
// GPU, resident from the code object's load until the process ends. Host code
// never passes this name to a kernel; it uses the device address looked up
// per device with hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[RB_STATIC_SCRATCH_BYTES];

constexpr int SCRATCH_MAX_DEVICES = 64;
std::mutex scratch_mu;
void* scratch_ptr[SCRATCH_MAX_DEVICES];
bool scratch_looked_up[SCRATCH_MAX_DEVICES];
}  // namespace

// Runtime support (not part of the C ABI): look up, once per device and with
// that device current, the device address of its copy of the scratch array.
rb_status rb_static_scratch_setup(int device) {
  if (device < 0 || device >= SCRATCH_MAX_DEVICES) return RB_EDEVICE;
  std::lock_guard<std::mutex> lk(scratch_mu);
  if (!scratch_looked_up[device]) {
    int cur = -1;
    if (hipGetDevice(&cur) != hipSuccess) return RB_EDEVICE;
    if (cur != device && hipSetDevice(device) != hipSuccess) return RB_EDEVICE;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != device) (void)hipSetDevice(cur);
    if (e != hipSuccess || !p) return RB_EDEVICE;
    scratch_ptr[device] = p;
    scratch_looked_up[device] = true;
  }
  return RB_OK;
}

// The device address of the device's scratch copy (nullptr before
// rb_static_scratch_setup succeeded on it).
void* rb_static_scratch(int device) {
  if (device < 0 || device >= SCRATCH_MAX_DEVICES) return nullptr;
  std::lock_guard<std::mutex> lk(scratch_mu);
  return scratch_looked_up[device] ? scratch_ptr[device] : nullptr;
}

// ---------------------------------------------------------------- cache scrub

namespace {
// Reads bytes of buf (a multiple of 16) so that L2 and the Infinity Cache hold
// only its clean lines afterwards; the loads feed a value stored only in a
// case that never happens, so they are not removed.
__global__ __launch_bounds__(256) void k_scrub(const u32x4_t* __restrict__ buf, int64_t n, unsigned* sink) {
  u32x4_t x = {0u, 0u, 0u, 0u};
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) x ^= buf[i];
  if (x.x == 0x9e3779b9u && x.y == 0x7f4a7c15u && x.z == 0xf39cc060u && x.w == 0x5cedc834u) sink[0] = 1u;
}
}  // namespace

// Cold-cache profiling support for the scheduler (not part of the C ABI).
void rb_scrub_caches(hipStream_t stream, const void* buf, size_t bytes, unsigned* sink) {
  hipLaunchKernelGGL(k_scrub, dim3(4096), dim3(256), 0, stream, (const u32x4_t*)buf, (int64_t)(bytes / 16), sink);
}

// ---------------------------------------------------------------- kernel ABI

extern "C" {

rb_status rb_k_route(void* stream, int32_t kind, const rb_k_batch* batches, int32_t n_batches,
                     const rb_k_req* reqs, int32_t n_reqs, const int32_t* lens, int64_t lens_len, int32_t d_in,
                     int32_t d_out, int32_t n_tables, rb_k_row* rows, int32_t n_rows_total, int64_t out_len,
                     int32_t* err) {
  if (n_batches < 0 || n_reqs < 0 || n_rows_total < 0 || lens_len < 0 || out_len < 0 || !batches || !rows ||
      !err || d_in < 1 || d_out < 1)
    return RB_EINVAL;
  if (n_reqs > 0 && !reqs) return RB_EINVAL;
  if (kind < RB_MODEL_MLP || kind > RB_MODEL_SEQPOOL) return RB_EINVAL;
  if (kind != RB_MODEL_MLP && !lens) return RB_EINVAL;
  if (kind == RB_MODEL_RANKING && (n_tables < 1 || n_tables > MAX_TABLES)) return RB_EINVAL;
  if (n_batches == 0) return RB_OK;
  hipLaunchKernelGGL(k_route, dim3(n_batches), dim3(256), 0, (hipStream_t)stream, kind, batches, reqs, n_reqs, lens,
                     lens_len, d_in, d_out, n_tables, rows, n_rows_total, out_len, err);
  return launch_status();
}

rb_status rb_k_assemble(void* stream, const rb_k_row* rows, int32_t n_rows_total, int32_t seq_T,
                        int32_t seq_real_only, const float* dense, int64_t dense_len, int32_t d_in, void* X,
                        int32_t ldx, int32_t out_bf16, float pad, int32_t* err) {
  if (n_rows_total < 0 || seq_T < 0 || d_in < 1 || ldx < d_in || (ldx & 7) || !rows || !X || !err)
    return RB_EINVAL;
  if (seq_real_only < 0 || seq_real_only > 2) return RB_EINVAL;
  if (seq_real_only && (seq_T == 0 || n_rows_total % seq_T || out_bf16)) return RB_EINVAL;
  if (n_rows_total == 0) return RB_OK;
  auto lg2 = [](int v) { int l = 0; while ((1 << l) < v) ++l; return (1 << l) == v ? l : -1; };
  if (seq_real_only) {
    const dim3 grid(n_rows_total / seq_T, (seq_T + SEQ_TOK - 1) / SEQ_TOK);
    if (seq_real_only == 2)
      hipLaunchKernelGGL(k_assemble_seq<true>, grid, dim3(256), 0, (hipStream_t)stream, rows, seq_T, dense, dense_len,
                         d_in, (float*)X, ldx, (int64_t)n_rows_total, err, lg2(ldx / 8));
    else
      hipLaunchKernelGGL(k_assemble_seq<false>, grid, dim3(256), 0, (hipStream_t)stream, rows, seq_T, dense,
                         dense_len, d_in, (float*)X, ldx, (int64_t)n_rows_total, err, lg2(ldx / 8));
    return launch_status();
  }
  const int64_t threads = (int64_t)n_rows_total * (ldx / 8);
  const unsigned g = blocks_for(threads);
  const int lg_c = lg2(ldx / 8), lg_t = seq_T > 0 ? lg2(seq_T) : 0;
  const bool pow2 = lg_c >= 0 && lg_t >= 0 && (int64_t)g * 256 < ((int64_t)1 << 31);
  hipStream_t hs = (hipStream_t)stream;
#define RB_ASM(B, P)                                                                                         \
  hipLaunchKernelGGL((k_assemble<B, P>), dim3(g), dim3(256), 0, hs, rows, n_rows_total, seq_T, dense, dense_len, \
                     d_in, X, ldx, pad, err, lg_c, lg_t)
  if (out_bf16) {
    if (pow2) RB_ASM(true, true);
    else RB_ASM(true, false);
  } else {
    if (pow2) RB_ASM(false, true);
    else RB_ASM(false, false);
  }
#undef RB_ASM
  return launch_status();
}

rb_status rb_k_embbag_dedup(void* stream, const rb_k_row* rows, int32_t n_rows_total, const int32_t* lens,
                            const int32_t* ids, int64_t ids_len, const void* const* tables, int32_t n_tables,
                            int64_t table_rows, int32_t emb_dim, const float* dense, int32_t n_dense, void* X,
                            int32_t ldx, float pad, int32_t* err) {
  if (emb_dim != EMB_DIM || n_tables < 1 || n_tables > MAX_TABLES || n_dense < 0 || n_dense > 256 ||
      table_rows < 1 || table_rows > INT32_MAX || ids_len < 0)
    return RB_EINVAL;
  if (n_rows_total < 0 || ldx < n_tables * EMB_DIM + n_dense || (ldx & 7) || !rows || !X || !err || !tables)
    return RB_EINVAL;
  if (n_rows_total == 0) return RB_OK;
  const unsigned grid = (unsigned)((n_rows_total + DD_ROWS - 1) / DD_ROWS) * n_tables;
  hipLaunchKernelGGL(k_embbag_dedup, dim3(grid), dim3(DD_NT), 0, (hipStream_t)stream, rows, n_rows_total, lens, ids,
                     ids_len, (const bf16_t* const*)tables, n_tables, table_rows, dense, n_dense, (bf16_t*)X, ldx,
                     pad, err);
  return launch_status();
}

rb_status rb_k_embbag(void* stream, const rb_k_row* rows, int32_t n_rows_total, const int32_t* lens,
                      const int32_t* ids, int64_t ids_len, const void* const* tables, int32_t n_tables,
                      int64_t table_rows, int32_t emb_dim, const float* dense, int32_t n_dense, void* X, int32_t ldx,
                      float pad, int32_t* err) {
  if (emb_dim != EMB_DIM || n_tables < 1 || n_tables > MAX_TABLES || n_dense < 0 || n_dense > 256 ||
      table_rows < 1 || ids_len < 0)
    return RB_EINVAL;
  if (n_rows_total < 0 || ldx < n_tables * EMB_DIM + n_dense || (ldx & 7) || !rows || !X || !err || !tables)
    return RB_EINVAL;
  if (n_rows_total == 0) return RB_OK;
  const int n_slices = std::min(EMB_SLICES, (int)n_tables);
  const int gpr = (n_tables + n_slices - 1) / n_slices;  // groups per row (bags of one slice)
  const int rpw = 32 / gpr;                              // rows per workgroup (32 groups)
  const unsigned grid = (unsigned)((n_rows_total + rpw - 1) / rpw) * n_slices;
  hipLaunchKernelGGL(k_embbag, dim3(grid), dim3(256), 0, (hipStream_t)stream, rows, n_rows_total, lens, ids, ids_len,
                     (const bf16_t* const*)tables, n_tables, table_rows, dense, n_dense, (bf16_t*)X, ldx, n_slices,
                     gpr, rpw, pad, err);
  return launch_status();
}

namespace {
rb_status gemm_bf16_impl(void* stream, const void* X, int32_t ldx, const void* W, int32_t ldw, const float* b,
                         void* Y, int32_t ldy, int32_t M, int32_t N, int32_t K, int32_t act, int32_t out_f32,
                         OutMap om) {
  if (M < 0 || N <= 0 || K <= 0 || (N % 128) || (K % G16_KALIGN) || ldx < K || ldw < K) return RB_EINVAL;
  if ((ldx & 7) || (ldw & 7) || !X || !W || !b) return RB_EINVAL;
  // operand byte offsets within a 256-row tile are 32-bit
  if ((int64_t)ldx * 512 >= ((int64_t)1 << 31) || (int64_t)ldw * 512 >= ((int64_t)1 << 31)) return RB_EINVAL;
  if (act != RB_ACT_NONE && act != RB_ACT_RELU && act != RB_ACT_SIGMOID) return RB_EINVAL;
  if (M == 0) return RB_OK;
  hipStream_t s = (hipStream_t)stream;
  const bf16_t* x = (const bf16_t*)X;
  const bf16_t* w = (const bf16_t*)W;
  // Tile shape, k-step, stage count and tile order only change speed: every
  // choice accumulates each output in the same k order with the same
  // instruction (identical bits). The largest tile that still gives every CU a
  // tile: 256 x 256 (k-step 64, 2 stages, 128 KB LDS, every row's k-step a
  // whole 128-byte line) as 4 waves of 128 x 128 when there are at least two
  // tiles per CU (half the fragment reads per flop of 8 waves of 64 x 128), as
  // 8 waves of 64 x 128 when fewer (two waves per SIMD hide more of the single
  // round's start and end), else 256 x 128 (8 waves of 64 x 64, k-step
  // 64, 3 stages, 144 KB), else
  // 128 x 128 (8 waves of 64 x 32, k-step 64, 4 stages, 128 KB), 128 x 64 (4
  // waves of 64 x 32, 96 KB) or 64 x 64 (2 waves of 64 x 32, 64 KB). XCD-contiguous
  // tile order when all of W fits in one XCD's L2 (each XCD then keeps its A
  // row-blocks and W in its own L2); plain order otherwise (contiguous ranges
  // would stream all of W through every XCD).
  //
  // With more 256 x 128 tiles than compute units, the grid is persistent (one
  // workgroup per CU, each taking every CU-count-th tile) when K is a multiple of the
  // stage count in k-steps: the operand loads then run on across tile
  // boundaries, so a tile's first k-steps load during the previous tile's last
  // steps and epilogue.
  const int64_t rows256 = (M + 255) / 256;
  const bool xcd = (int64_t)N * K * 2 <= (4 << 20);
  const unsigned cus = device_cus() & ~7u;
#define RB_PICK(BM, BN, WM, WN, NT, BK, S, P)                                                                   \
  do {                                                                                                          \
    if (xcd)                                                                                                    \
      launch_gemm_bf16<BM, BN, WM, WN, NT, BK, S, 1, P>(s, x, ldx, w, ldw, b, Y, ldy, M, N, K, act, out_f32, cus, om); \
    else                                                                                                        \
      launch_gemm_bf16<BM, BN, WM, WN, NT, BK, S, 0, P>(s, x, ldx, w, ldw, b, Y, ldy, M, N, K, act, out_f32, cus, om); \
  } while (0)
  auto persist = [&](int bm, int bn, int bk, int st) {
    const int64_t tiles = ((M + bm - 1) / bm) * (int64_t)(N / bn);
    const int nk = K / bk;
    return cus >= 8 && tiles > (int64_t)cus && nk >= st && nk % st == 0;
  };
  if (N % 256 == 0 && rows256 * (N / 256) >= 256) {
    if (rows256 * (N / 256) >= 2 * (int64_t)cus)
      RB_PICK(256, 256, 128, 128, 256, 64, 2, false);
    else
      RB_PICK(256, 256, 64, 128, 512, 64, 2, false);
  } else if (rows256 * (N / 128) >= 256) {
    if (persist(256, 128, 64, 3))
      RB_PICK(256, 128, 64, 64, 512, 64, 3, true);
    else
      RB_PICK(256, 128, 64, 64, 512, 64, 3, false);
  } else {
    // fewer tiles than that: the k-loop's latency bounds a launch of a few
    // batches, so the largest of 128 x 128, 128 x 64 and 64 x 64 tiles that
    // still gives half the compute units a tile (512 x 1024 x 1728: 12.5 ->
    // 8.7 us with 64 x 64; 2816 x 512 x 1024: 9.7 -> 7.3 us with 128 x 64)
    const int64_t rows128 = (M + 127) / 128, half = std::max<int64_t>(cus / 2, 1);
    if (rows128 * (N / 128) >= half)
      RB_PICK(128, 128, 64, 32, 512, 64, 4, false);
    else if (rows128 * (N / 64) >= half)
      RB_PICK(128, 64, 64, 32, 256, 64, 4, false);
    else
      RB_PICK(64, 64, 64, 32, 128, 64, 4, false);
  }
#undef RB_PICK
  return launch_status();
}
}  // namespace

rb_status rb_k_gemm_bf16(void* stream, const void* X, int32_t ldx, const void* W, int32_t ldw, const float* b,
                         void* Y, int32_t ldy, int32_t M, int32_t N, int32_t K, int32_t act, int32_t out_f32) {
  if (ldy < N || (ldy & 7) || ((uintptr_t)Y & 15) || !Y) return RB_EINVAL;
  return gemm_bf16_impl(stream, X, ldx, W, ldw, b, Y, ldy, M, N, K, act, out_f32, OutMap{});
}

rb_status rb_k_gemm_bf16_rows(void* stream, const void* X, int32_t ldx, const void* W, int32_t ldw, const float* b,
                              int32_t M, int32_t N, int32_t K, int32_t act, const rb_k_row* rows, int32_t d_out,
                              float* out) {
  if (!rows || !out || d_out < 1 || d_out > N) return RB_EINVAL;
  return gemm_bf16_impl(stream, X, ldx, W, ldw, b, nullptr, N, M, N, K, act, 1, OutMap{rows, out, d_out});
}

namespace {
rb_status gemm_f32_impl(void* stream, const float* X, int32_t ldx, const float* W, int32_t ldw, const float* b,
                        float* Y, int32_t ldy, int32_t M, int32_t N, int32_t K, int32_t act,
                        const rb_k_row* skip_rows, int32_t skip_T, OutMap om) {
  if (M < 0 || N <= 0 || K <= 0 || (N % 64) || (K % G32_KALIGN) || ldx < K || ldw < K) return RB_EINVAL;
  if ((ldx & 3) || (ldw & 3) || !X || !W || !b) return RB_EINVAL;
  if (((uintptr_t)X & 15) || ((uintptr_t)W & 15)) return RB_EINVAL;
  // operand byte offsets within a 64-row tile are 32-bit
  if ((int64_t)ldx * 4 * G32_BM >= ((int64_t)1 << 31) || (int64_t)ldw * 4 * 64 >= ((int64_t)1 << 31)) return RB_EINVAL;
  if (act != RB_ACT_NONE && act != RB_ACT_RELU && act != RB_ACT_SIGMOID) return RB_EINVAL;
  if (skip_rows && (skip_T <= 0 || skip_T % G32_BM)) return RB_EINVAL;
  if (M == 0) return RB_OK;
  hipStream_t s = (hipStream_t)stream;
  // 64 x 64 tiles (64 rows: the padding-token skip granularity), 4 waves of
  // 32 x 32, k-step 16, 3 stages (24 KB LDS, six workgroups per CU). Small
  // wave tiles keep the work per wave small, so the CUs stay evenly loaded when
  // padding-token blocks leave holes in the grid (64 x 64 wave tiles measured
  // up to 1.5x slower there). XCD-contiguous tile order when W fits in one
  // XCD's L2 (each XCD then reads its X rows once; plain order measured 1.5x
  // slower on sequence groups).
  const bool xcd = (int64_t)N * K * 4 <= (4 << 20);
  if (xcd)
    launch_gemm<float, G32_BM, 64, 32, 32, 256, 64, 3, 1>(s, X, ldx, W, ldw, b, Y, ldy, M, N, K, act, true, skip_rows,
                                                          skip_T, 0, om);
  else
    launch_gemm<float, G32_BM, 64, 32, 32, 256, 64, 3, 0>(s, X, ldx, W, ldw, b, Y, ldy, M, N, K, act, true, skip_rows,
                                                          skip_T, 0, om);
  return launch_status();
}
}  // namespace

rb_status rb_k_gemm_f32(void* stream, const float* X, int32_t ldx, const float* W, int32_t ldw, const float* b,
                        float* Y, int32_t ldy, int32_t M, int32_t N, int32_t K, int32_t act,
                        const rb_k_row* skip_rows, int32_t skip_T) {
  if (ldy < N || (ldy & 3) || ((uintptr_t)Y & 15) || !Y) return RB_EINVAL;
  return gemm_f32_impl(stream, X, ldx, W, ldw, b, Y, ldy, M, N, K, act, skip_rows, skip_T, OutMap{});
}

rb_status rb_k_gemm_f32_rows(void* stream, const float* X, int32_t ldx, const float* W, int32_t ldw, const float* b,
                             int32_t M, int32_t N, int32_t K, int32_t act, const rb_k_row* rows, int32_t d_out,
                             float* out) {
  if (!rows || !out || d_out < 1 || d_out > N) return RB_EINVAL;
  return gemm_f32_impl(stream, X, ldx, W, ldw, b, nullptr, N, M, N, K, act, nullptr, 0, OutMap{rows, out, d_out});
}

rb_status rb_k_head(void* stream, const rb_k_row* rows, int32_t n_rows_total, const void* H, int32_t ldh,
                    const void* w, float b, int32_t K, int32_t act, float* out) {
  if (n_rows_total < 0 || K < 1 || ldh < K || !rows || !H || !w || !out) return RB_EINVAL;
  if (act != RB_ACT_NONE && act != RB_ACT_SIGMOID) return RB_EINVAL;
  if (n_rows_total == 0) return RB_OK;
  const unsigned g = (unsigned)((n_rows_total + 15) / 16);
  // 16-byte loads when every row and the weight vector start 16-byte aligned
  const int vec = (K % 8 == 0) && (ldh % 8 == 0) && ((uintptr_t)H % 16 == 0) && ((uintptr_t)w % 16 == 0);
  if (act == RB_ACT_SIGMOID)
    hipLaunchKernelGGL(k_head<RB_ACT_SIGMOID>, dim3(g), dim3(256), 0, (hipStream_t)stream, rows, n_rows_total,
                       (const bf16_t*)H, ldh, (const bf16_t*)w, b, K, vec, out);
  else
    hipLaunchKernelGGL(k_head<RB_ACT_NONE>, dim3(g), dim3(256), 0, (hipStream_t)stream, rows, n_rows_total,
                       (const bf16_t*)H, ldh, (const bf16_t*)w, b, K, vec, out);
  return launch_status();
}

rb_status rb_k_gemm_head(void* stream, const void* X, int32_t ldx, const void* W, int32_t ldw, const float* b,
                         int32_t M, int32_t K, int32_t act, const rb_k_row* rows, const void* w_head, float b_head,
                         int32_t head_act, float* out) {
  if (M < 0 || K <= 0 || (K % G16_KALIGN) || ldx < K || ldw < K || (ldx & 7) || (ldw & 7)) return RB_EINVAL;
  if (!X || !W || !b || !rows || !w_head || !out || ((uintptr_t)w_head & 15)) return RB_EINVAL;
  if ((int64_t)ldx * 512 >= ((int64_t)1 << 31) || (int64_t)ldw * 512 >= ((int64_t)1 << 31)) return RB_EINVAL;
  if (act != RB_ACT_NONE && act != RB_ACT_RELU && act != RB_ACT_SIGMOID) return RB_EINVAL;
  if (head_act != RB_ACT_NONE && head_act != RB_ACT_SIGMOID) return RB_EINVAL;
  if (M == 0) return RB_OK;
  // 128 x 256 tiles (every row's 256 outputs in one workgroup), 8 waves of
  // 64 x 64 (two per SIMD: 4 waves of 64 x 128 measured 16% slower), k-step
  // 64, 3 stages; XCD-contiguous order (W is 256 x K bf16). With fewer such
  // tiles than half the compute units (a launch of a few batches, bound by
  // its k-loop's latency), 64 x 256 tiles of 8 waves of 64 x 32.
  const bool small = (int64_t)(M + 127) / 128 < std::max<int64_t>(device_cus() / 2, 1);
  const unsigned g = (unsigned)(small ? (M + 63) / 64 : (M + 127) / 128);
  const HeadArgs ha{rows, (const bf16_t*)w_head, b_head, out};
  hipStream_t s = (hipStream_t)stream;
#define RB_GH(A, H)                                                                                                    \
  do {                                                                                                                 \
    if (small)                                                                                                         \
      hipLaunchKernelGGL((k_gemm_head<64, 256, 64, 32, 512, 128, 3, 1, A, H>), dim3(g), dim3(512), 0, s,             \
                         (const bf16_t*)X, ldx, (const bf16_t*)W, ldw, b, M, K, ha);                                   \
    else                                                                                                               \
      hipLaunchKernelGGL((k_gemm_head<128, 256, 64, 64, 512, 128, 3, 1, A, H>), dim3(g), dim3(512), 0, s,            \
                         (const bf16_t*)X, ldx, (const bf16_t*)W, ldw, b, M, K, ha);                                   \
  } while (0)
  if (head_act == RB_ACT_SIGMOID) {
    if (act == RB_ACT_RELU) RB_GH(RB_ACT_RELU, RB_ACT_SIGMOID);
    else if (act == RB_ACT_SIGMOID) RB_GH(RB_ACT_SIGMOID, RB_ACT_SIGMOID);
    else RB_GH(RB_ACT_NONE, RB_ACT_SIGMOID);
  } else {
    if (act == RB_ACT_RELU) RB_GH(RB_ACT_RELU, RB_ACT_NONE);
    else if (act == RB_ACT_SIGMOID) RB_GH(RB_ACT_SIGMOID, RB_ACT_NONE);
    else RB_GH(RB_ACT_NONE, RB_ACT_NONE);
  }
#undef RB_GH
  return launch_status();
}

rb_status rb_k_mlp_tail(void* stream, const rb_k_row* rows, int32_t n_rows_total, const void* H1, int32_t ldh1,
                        int32_t K2, const void* W2, int32_t ldw2, const float* b2, const void* W3, int32_t ldw3,
                        const float* b3, const void* w4, float b4, int32_t act, float* out) {
  if (n_rows_total < 0 || K2 < MT_KS || K2 % MT_KS || ldh1 < K2 || ldw2 < K2 || ldw3 < MT_N2) return RB_EINVAL;
  if ((ldh1 & 7) || (ldw2 & 7) || (ldw3 & 7) || !rows || !H1 || !W2 || !b2 || !W3 || !b3 || !w4 || !out)
    return RB_EINVAL;
  if (((uintptr_t)H1 & 15) || ((uintptr_t)W2 & 15) || ((uintptr_t)W3 & 15) || ((uintptr_t)w4 & 15)) return RB_EINVAL;
  if (act != RB_ACT_NONE && act != RB_ACT_SIGMOID) return RB_EINVAL;
  if (n_rows_total == 0) return RB_OK;
  const unsigned g = (unsigned)((n_rows_total + MT_BM - 1) / MT_BM);
  if (act == RB_ACT_SIGMOID)
    hipLaunchKernelGGL(k_mlp_tail<RB_ACT_SIGMOID>, dim3(g), dim3(MT_NT), 0, (hipStream_t)stream, (const bf16_t*)H1,
                       ldh1, K2, (const bf16_t*)W2, ldw2, b2, (const bf16_t*)W3, ldw3, b3, (const bf16_t*)w4, b4, rows,
                       n_rows_total, out);
  else
    hipLaunchKernelGGL(k_mlp_tail<RB_ACT_NONE>, dim3(g), dim3(MT_NT), 0, (hipStream_t)stream, (const bf16_t*)H1,
                       ldh1, K2, (const bf16_t*)W2, ldw2, b2, (const bf16_t*)W3, ldw3, b3, (const bf16_t*)w4, b4, rows,
                       n_rows_total, out);
  return launch_status();
}

rb_status rb_k_seqpool(void* stream, const rb_k_row* rows, int32_t n_seqs, int32_t seq_T, int64_t packed_rows,
                       const float* H, int32_t ldh, int32_t D, const float* Wh, const float* bh, int32_t n_out,
                       int32_t act, float* out) {
  if (n_seqs < 0 || seq_T < 1 || packed_rows < 0 || D < 1 || D > POOL_MAX_D || ldh < D || n_out < 1 ||
      n_out > POOL_MAX_OUT)
    return RB_EINVAL;
  if (act != RB_ACT_NONE && act != RB_ACT_SOFTMAX) return RB_EINVAL;
  if (!rows || !H || !Wh || !bh || !out) return RB_EINVAL;
  if (n_seqs == 0) return RB_OK;
  hipLaunchKernelGGL(k_seqpool, dim3(n_seqs), dim3(256), 0, (hipStream_t)stream, rows, n_seqs, seq_T, packed_rows, H,
                     ldh, D, Wh, bh, n_out, act, out);
  return launch_status();
}

rb_status rb_k_split(void* stream, const rb_k_row* rows, int32_t n_rows_total, const float* Y, int32_t ldy,
                     int32_t d_out, float* out) {
  if (n_rows_total < 0 || d_out < 1 || ldy < d_out || !rows || !Y || !out) return RB_EINVAL;
  if (n_rows_total == 0) return RB_OK;
  // 16-byte path: width, row stride and both bases multiples of 4 floats
  const bool v4 = (d_out % 4) == 0 && (ldy % 4) == 0 && ((uintptr_t)Y % 16) == 0 && ((uintptr_t)out % 16) == 0;
  const int per = v4 ? d_out / 4 : d_out;
  int tpr = 1;
  while (tpr < per && tpr < 256) tpr <<= 1;
  const unsigned g = (unsigned)((n_rows_total + 256 / tpr - 1) / (256 / tpr));
  if (v4)
    hipLaunchKernelGGL(k_split<4>, dim3(g), dim3(256), 0, (hipStream_t)stream, rows, n_rows_total, tpr, Y, ldy,
                       d_out, out);
  else
    hipLaunchKernelGGL(k_split<1>, dim3(g), dim3(256), 0, (hipStream_t)stream, rows, n_rows_total, tpr, Y, ldy,
                       d_out, out);
  return launch_status();
}

}  // extern "C"
