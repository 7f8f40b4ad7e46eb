"""CPU oracle (test infrastructure): see higgs_oracle."""
