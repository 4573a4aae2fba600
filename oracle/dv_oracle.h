/* CPU oracle for the KV-cache streaming path.  TEST INFRASTRUCTURE ONLY:
 * only the tests, the smoke check and the benchmark's CPU-baseline leg may
 * load it.  It shares no code with the HIP library.
 *
 * What it computes (all bit copies; elements are opaque elem_bytes words, no
 * arithmetic is applied to them):
 *
 *   pack    the non-contiguous region of a KV cache selected by a layer range
 *           [l0,l1) and per-sequence token ranges [t0_b,t1_b) -> one
 *           contiguous buffer (the paper's buffered copy into a temporary GPU
 *           buffer, Sec. 4.1.1 optimisation 1; the scatter primitive of
 *           Table 1);
 *   unpack  the inverse, into a receiver's layout (gather/fetch of Table 1;
 *           restoring a lost cache from its replica, Sec. 4.2.3); every byte
 *           outside the selected region stays as it was;
 *   copy    the same region between two layouts at equal logical coordinates
 *           (microbatch swapping between GPU slots and host memory,
 *           Sec. 4.2.2).
 *
 * Logical element X(l, kv, b, h, s, d): layer l, kv = 0 key / 1 value,
 * sequence b, head h, token s, dimension d.  Storage index by layout:
 *   dense  ((((l*2+kv)*B + b)*H + h)*S + s)*D + d
 *   paged  ((((l*2+kv)*NB + BT[b][s/bs])*H + h)*bs + s%bs)*D + d
 *   ksplit key slab (kv=0): (((((l*2)*B + b)*H + h)*(D/x) + d/x)*S + s)*x + d%x
 *          with x = 16/elem_bytes; the value slab (kv=1) is dense.
 * Wire (contiguous buffer), with n_b = t1_b - t0_b, P_b = sum_{b'<b} n_b',
 * N = sum_b n_b:
 *   W = ((l-l0)*2+kv)*N*H*D + P_b*H*D + h*n_b*D + (s-t0_b)*D + d
 * i.e. [layer][K|V][sequence][head][token][dim] with ragged sequences.
 */
#ifndef DV_ORACLE_H
#define DV_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { DVO_DENSE = 0, DVO_PAGED = 1, DVO_KSPLIT = 2 };
enum { DVO_OK = 0, DVO_INVALID = -1, DVO_RANGE = -2 };

typedef struct {
  int32_t kind;
  int64_t elem_bytes;
  int64_t layers, heads, head_dim, batch;
  int64_t seq_cap;                 /* dense / ksplit: S */
  int64_t block_size, num_blocks;  /* paged: bs, NB */
  int64_t max_blocks;              /* paged: columns of the block table */
  const int32_t* block_table;      /* paged: host [batch][max_blocks] */
} dvo_layout;

/* Storage element index of X(l,kv,b,h,s,d), or -1 if it has no storage
 * (token beyond capacity, or a paged table entry outside [0, NB)). */
int64_t dvo_elem_index(const dvo_layout* c, int64_t l, int64_t kv, int64_t b, int64_t h,
                       int64_t s, int64_t d);

/* Total storage elements of the layout (dense: L*2*B*H*S*D; paged:
 * L*2*NB*H*bs*D). */
int64_t dvo_storage_elems(const dvo_layout* c);

/* DVO_OK, DVO_INVALID (bad shape) or DVO_RANGE (layer or token range outside
 * the layout, or a paged range touching an invalid table entry). */
int dvo_check(const dvo_layout* c, int64_t l0, int64_t l1, const int32_t* t0, const int32_t* t1);

/* Elements of the wire for these ranges: (l1-l0)*2*H*D*N. */
int64_t dvo_wire_elems(const dvo_layout* c, int64_t l0, int64_t l1, const int32_t* t0,
                       const int32_t* t1);

int dvo_pack(const dvo_layout* c, const void* cache, int64_t l0, int64_t l1, const int32_t* t0,
             const int32_t* t1, void* wire);
int dvo_unpack(const dvo_layout* c, void* cache, int64_t l0, int64_t l1, const int32_t* t0,
               const int32_t* t1, const void* wire);
/* dst[X] = src[X] for every X in the ranges; src and dst may differ in kind
 * and capacity but must agree on layers, heads, head_dim, batch, elem_bytes. */
int dvo_copy_ranges(const dvo_layout* src_l, const void* src, const dvo_layout* dst_l, void* dst,
                    int64_t l0, int64_t l1, const int32_t* t0, const int32_t* t1);
/* For each wire element index w[i], the storage index of the element it
 * holds (-1 for an index outside the wire). */
int dvo_wire_to_storage(const dvo_layout* c, int64_t l0, int64_t l1, const int32_t* t0,
                        const int32_t* t1, const int64_t* w, int64_t n, int64_t* out);

#ifdef __cplusplus
}
#endif
#endif
