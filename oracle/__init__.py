"""Plain float64 CPU oracle of the AS2D target verification step.

TEST INFRASTRUCTURE ONLY.  Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import it.  The product path (the HIP
library and its Python binding) never imports, calls or links anything
here, and the oracle imports nothing from the product path: the two share
only the seeded input generators in workload/.
"""
from .model import OracleModel, greedy, rms_norm, rope, silu, attention, verify_block
from .align import CandidateBuffer, ReadCursor, decode_with_buffer
