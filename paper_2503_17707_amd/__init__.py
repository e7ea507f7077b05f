"""MI355X cold-start prefill (PipeBoost, arXiv 2503.17707): layer-streamed
OPT prefill with unmerged multi-adapter LoRA, behind the C ABI of
libpipeboost.so.  ``binding`` marshals arguments; the HIP library does the work.
"""
from . import binding  # noqa: F401
