"""Seeded synthetic inputs (weights, contexts, synthetic K/V, draft
corruption draws) shared by the oracle and the GPU path.  Holds none of the
verification method's arithmetic."""
