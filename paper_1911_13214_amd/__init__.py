"""MI355X (gfx950) solver for optimal persistent activation checkpointing on
heterogeneous chains (Beaumont et al., arXiv 1911.13214).

``rotor`` binds the C ABI of include/rotor.h; ``chaingen`` draws seeded
synthetic chains.  Importing the package loads nothing."""
