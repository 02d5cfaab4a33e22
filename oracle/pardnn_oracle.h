/*
 * pardnn_oracle.h -- sequential CPU oracle (test infrastructure only).
 *
 * Host arrays only. Node ids are 0..n_nodes-1; edge e runs src[e] -> dst[e].
 * Every function returns ORC_OK or a negative status and writes its outputs
 * only on success. Definitions follow the paper's Table 2 (tl, bl, w_lvl,
 * CP); see pardnn_oracle.c for the readings taken where the paper is silent.
 */
#ifndef PARDNN_ORACLE_H
#define PARDNN_ORACLE_H

#include <stdint.h>

#define ORC_OK 0
#define ORC_E_INVAL (-1)
#define ORC_E_CYCLE (-2)
#define ORC_E_OVERFLOW (-3)
#define ORC_E_NOMEM (-4)

#ifdef __cplusplus
extern "C" {
#endif

int orc_validate(int32_t n_nodes, int64_t n_edges, const int32_t *src,
                 const int32_t *dst, const int64_t *comp,
                 const int64_t *edge_cost, const int64_t *mem);

int orc_levelize(int32_t n_nodes, int64_t n_edges, const int32_t *src,
                 const int32_t *dst, int32_t *level, int32_t *order,
                 int32_t *level_ptr /* [n_nodes + 1] */, int32_t *n_levels);

int orc_tb_levels(int32_t n_nodes, int64_t n_edges, const int32_t *src,
                  const int32_t *dst, const int64_t *comp,
                  const int64_t *edge_cost, const int32_t *label, int64_t *tl,
                  int64_t *bl, int64_t *makespan);

int orc_critical_path(int32_t n_nodes, int64_t n_edges, const int32_t *src,
                      const int32_t *dst, const int64_t *comp,
                      const int64_t *edge_cost, const int32_t *label,
                      const int64_t *tl, const int64_t *bl, int64_t makespan,
                      uint8_t *is_critical, int32_t *path, int32_t *path_len);

int orc_label_memory(int32_t n_nodes, const int64_t *mem, const int32_t *label,
                     int32_t n_labels, const int64_t *capacity,
                     int64_t *label_mem, int64_t *overflow);

#ifdef __cplusplus
}
#endif

#endif
