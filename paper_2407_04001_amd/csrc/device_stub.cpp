// The device runtime of a host-only build of libpase (no HIP): used only by
// the sanitizer build of the host code, which the CPU test suite runs under
// AddressSanitizer and UBSan.  Every call that would need a GPU fails with
// PASE_ERR_HIP; planning, validation and the launch image run as usual.
#include "internal.h"

namespace pase {

static pase_status no_device(pase_graph_t g) {
    return fail(g, PASE_ERR_HIP, "host-only build: no device runtime");
}

void device_release(pase_graph_t) {}
pase_status device_search(pase_graph_t g, void *, uint64_t *, uint32_t *) { return no_device(g); }
pase_status device_search_noalloc(pase_graph_t g, void *, uint64_t *, uint32_t *) { return no_device(g); }
pase_status device_table_entry(pase_graph_t g, int, uint64_t, uint64_t *, uint32_t *) { return no_device(g); }
pase_status device_fingerprint(pase_graph_t g, int, uint64_t *, uint64_t *) { return no_device(g); }
pase_status device_layer_costs(pase_graph_t g, uint32_t, uint64_t *) { return no_device(g); }
pase_status device_edge_costs(pase_graph_t g, uint32_t, uint64_t *) { return no_device(g); }

}  // namespace pase
