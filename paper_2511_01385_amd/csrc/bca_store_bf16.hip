// bca_store_bf16.hip -- the fused layer kernels of bca_kernels.hpp for StoreBF16 rows.
#include "bca_kernels.hpp"

namespace rdfft {

BcaStoreTables bca_tables_bf16() { return make_store_tables<StoreBF16>(); }

}  // namespace rdfft
