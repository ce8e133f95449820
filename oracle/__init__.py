"""CPU fp64 oracle of the Muon step (test infrastructure only; see muon_ref)."""
