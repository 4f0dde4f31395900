// Internal declarations shared by the libmgn host sources.
#pragma once
#include <stdint.h>

#include <string>

#include "../../include/mgn.h"

namespace mgn {

mgn_status partition_slabs(const int32_t* key, int64_t n, int32_t nparts, int32_t* part, std::string& err);
mgn_status graph_sizes(const int32_t* send, const int32_t* recv, int64_t n_edges, const int32_t* part,
                       int64_t n_nodes, int32_t p, int64_t* sizes, std::string& err);
mgn_status graph_build(const int32_t* send, const int32_t* recv, int64_t n_edges, const int32_t* part,
                       int64_t n_nodes, int32_t p, int32_t* row_ptr, int32_t* send_local, int32_t* eperm,
                       int32_t* trow_ptr, int32_t* tedge, int32_t* l2g, std::string& err);
mgn_status halo_masks(const int32_t* l2g_p, int64_t n_owned_p, int64_t n_halo_p, const int32_t* part,
                      int64_t n_nodes, const int32_t* l2g_q, int64_t n_owned_q, int32_t q, int32_t* recv_idx,
                      int32_t* send_rows, int64_t* count, std::string& err);
// Records msg as the model's last error (or the thread's, for a NULL model)
// and returns s.
mgn_status set_error(mgn_model* m, mgn_status s, const std::string& msg);
// Whether launch timing (mgn_timing_enable) is on for the model.
bool timing_enabled(const mgn_model* m);
mgn_status graph_check(int64_t no, int64_t nh, int64_t ne, const int32_t* row_ptr, const int32_t* send,
                       const int32_t* trow, const int32_t* tedge, std::string& err);

}  // namespace mgn
