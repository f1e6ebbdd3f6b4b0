// bca_store_f32.hip -- the fused layer kernels of bca_kernels.hpp for StoreF32 rows.
#include "bca_kernels.hpp"

namespace rdfft {

BcaStoreTables bca_tables_f32() { return make_store_tables<StoreF32>(); }

}  // namespace rdfft
